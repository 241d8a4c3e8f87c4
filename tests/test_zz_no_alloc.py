"""toc_left_mul_noalloc (the left product with its workspace in the library's static
device buffer) against toc_left_mul with a caller-allocated workspace: the same
result bit for bit (each output element is summed in one fixed order), on two calls
in a row, the second with a smaller input, so the second call runs on the buffer
the first call left behind."""

import ctypes as C

import numpy as np
import pytest

import paper_1702_06943_amd as T
from workloads import Batches, config_batches, config_G

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _upload(B):
    encs = T.toc_encode_batches(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    buf = torch.empty(T.toc_upload_size(encs), dtype=torch.uint8, device=DEV)
    dev = T.toc_upload(encs, buf)
    return dev, buf, T.toc_dev_info_get(dev)


def _both(dev, info, G, accumulate=False, init=None):
    """(toc_left_mul with its own workspace, toc_left_mul_noalloc called through
    the C ABI) on the same inputs."""
    k = G.shape[1]
    Gd = torch.from_numpy(np.ascontiguousarray(G)).to(DEV)
    rows_out = info["n_batches"] * info["n_cols"]
    outs = []
    for noalloc in (False, True):
        out = (torch.from_numpy(init).to(DEV) if init is not None
               else torch.full((rows_out, k), float("nan"), device=DEV))
        if noalloc:
            st = T.lib().toc_left_mul_noalloc(dev.handle, C.c_void_p(Gd.data_ptr()), k, k,
                                              C.c_void_p(out.data_ptr()), k, int(accumulate),
                                              C.c_void_p(torch.cuda.current_stream().cuda_stream))
            assert st == 0, T.lib().toc_last_error()
        else:
            ws_n, _ = T.toc_workspace_size(dev, T.TOC_OP_LEFT, k)
            ws = torch.empty(max(ws_n, 4) // 4, device=DEV) if ws_n else None
            T.toc_left_mul(dev, Gd, out, accumulate, ws)
        torch.cuda.synchronize()
        outs.append(out.cpu().numpy())
    return outs


def test_noalloc_equals_left_mul_two_calls():
    # call 1: 48 dense quantised batches at k = 64; the full grid's workspace
    # (one 3.8 MB slot per worker) is beyond the static buffer, so fewer workers run
    B1 = config_batches("c4", 0, 48)
    dev1, buf1, info1 = _upload(B1)
    ws_n, _ = T.toc_workspace_size(dev1, T.TOC_OP_LEFT, 64)
    assert ws_n > T.TOC_NOALLOC_SCRATCH_BYTES
    G1 = config_G("c4", 0, 48, 64)
    a, b = _both(dev1, info1, G1)
    assert not np.isnan(a).any()
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    del dev1, buf1
    # call 2, smaller: 6 image-like batches at k = 300 (5 column tiles), accumulating
    # into a given block
    B2 = config_batches("c3", 40, 6)
    dev2, buf2, info2 = _upload(B2)
    G2 = config_G("c3", 40, 6, 300)
    init = np.random.default_rng(3).standard_normal((6 * B2.n_cols, 300)).astype(np.float32)
    a, b = _both(dev2, info2, G2, accumulate=True, init=init)
    assert not np.isnan(a).any()
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_noalloc_rejects_beyond_the_buffer():
    """One batch of 1,500 dense quantised rows at k = 512: its G rows do not fit in
    LDS (fallback path) and its tree rows need more than the static buffer holds:
    TOC_EUNSUPPORTED, nothing launched."""
    parts = config_batches("c4", 0, 6)
    one = Batches(parts.n_cols, [int(parts.n_rows.sum())], parts.rowptr, parts.col, parts.val)
    dev, buf, info = _upload(one)
    ws_n, ws_min = T.toc_workspace_size(dev, T.TOC_OP_LEFT, 512)
    assert ws_min > T.TOC_NOALLOC_SCRATCH_BYTES
    G = torch.zeros((info["n_rows"], 512), device=DEV)
    out = torch.zeros((info["n_cols"], 512), device=DEV)
    with pytest.raises(T.TocError) as ei:
        T.toc_left_mul_noalloc(dev, G, out)
    assert ei.value.status == T.TOC_EUNSUPPORTED
