"""The device image written by toc_upload (built range of batches by range of
batches through two pinned staging buffers of 256 MiB) equals, array by array and
bit for bit, the image the same encodings give with TOC_UPLOAD_HOST (built in one
piece on the host).  900 image-like batches make about 680 MB, so the upload takes
three ranges and both staging buffers are reused."""

import numpy as np
import pytest

import paper_1702_06943_amd as T
from workloads import config_batches, tiny_batch, Batches

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _arrays(layout, info, bt):
    """(name, byte offset, byte length) of every array of the image."""
    nb = len(bt)
    n_codes, n_d = int(info["n_stored"]), int(info["n_codes"])
    tree = int((bt["n_int1"] + bt["n_codes"] - bt["n_lvl1"]).sum()) if nb else 0
    levels = int((bt["n_levels"] + 1).sum()) if nb else 0
    spans = int((bt["n_rows"] + 1).sum()) if nb else 0
    m = int(info["n_cols"])
    dt = int(np.maximum(1, (bt["n_d"].astype(np.int64) + 1023) // 1024).sum()) if nb else 0
    return [("batches", layout["batches"], 96 * nb), ("level", layout["level"], 4 * levels),
            ("key", layout["key"], 8 * n_codes), ("link", layout["link"], 8 * int(info["n_deep"])),
            ("span", layout["span"], 4 * spans), ("dcodes", layout["dcodes"], 4 * n_d),
            ("occ_off", layout["occ_off"], 4 * (n_codes + 2 * nb)),
            ("tlist", layout["tlist"], 4 * tree),
            ("dtiles", layout["dtiles"], 16 * dt), ("cols", layout["cols"], 16 * nb * (m + 1)),
            ("tchild", layout["tchild"], 4 * (tree + nb)),
            ("centry", layout["centry"], 4 * (n_d + tree)),
            ("cval", layout["cval"], 4 * (n_d + tree))]


@pytest.mark.parametrize("case", ["image_like_900", "tiny_mixed"])
def test_chunked_upload_equals_host_image(case):
    if case == "image_like_900":
        B = config_batches("c3", 21, 900)
    else:
        parts = []
        for i, spec in enumerate([dict(n_rows=30, density=0.5, n_values=3, prefix_copy=0.6),
                                  dict(n_rows=0, density=0.5, n_values=2),
                                  dict(n_rows=4, density=0.0, n_values=2),
                                  dict(n_rows=1, density=1.0, n_values=1)]):
            rp, c, v = tiny_batch(500 + i, n_cols=50, zeros=True, **spec)
            parts.append(Batches(50, [spec["n_rows"]], rp, c, v))
        B = Batches.concat(parts)
    encs = T.toc_encode_batches(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    size = T.toc_upload_size(encs)
    host = np.zeros(size, np.uint8)
    hd = T.toc_upload(encs, host, T.TOC_UPLOAD_HOST)
    buf = torch.full((size,), 0xAB, dtype=torch.uint8, device=DEV)
    dd = T.toc_upload(encs, buf)
    dev = buf.cpu().numpy()
    layout = T.toc_dev_layout_get(dd)
    assert layout == T.toc_dev_layout_get(hd)
    info = T.toc_dev_info_get(dd)
    bt = np.frombuffer(host[layout["batches"]:layout["batches"] + 96 * info["n_batches"]].tobytes(),
                       dtype=T.BATCH_DTYPE)
    for name, off, n in _arrays(layout, info, bt):
        assert np.array_equal(dev[off:off + n], host[off:off + n]), name
    if case == "image_like_900":
        assert size > 512 << 20        # three staging ranges
