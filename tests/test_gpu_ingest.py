"""GPU parity of the upload image built on the device from physical bytes (section
3.2's packed (I, D), read back as in section 4.1.1, C' by Algorithm 2) with the
image toc_upload builds on the host from the same batches: the two buffers must be
equal byte for byte, and the products and decode on the device-built image equal
those on the host-built one bit for bit and the oracle within 1e-5 * S (decode
exactly)."""

import numpy as np
import pytest

import oracle as O
import paper_1702_06943_amd as T
from workloads import Batches, config_batches, tiny_batch

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"
TOL = 1e-5


def _blobs(encs):
    blobs = [T.toc_enc_pack(e) for e in encs]
    infos = [T.toc_phys_info_get(b) for b in blobs]
    off = np.concatenate([[0], np.cumsum([len(b) for b in blobs])]).astype(np.int64)
    cat = np.concatenate([np.asarray(b, np.uint8) for b in blobs] + [np.zeros(1, np.uint8)])
    return torch.from_numpy(cat).to(DEV), off, infos


def _ingest(encs, n_cols, ws_bytes=None):
    dblob, off, infos = _blobs(encs)
    full, least = T.toc_ingest_workspace_size(infos, n_cols)
    nb = full if ws_bytes is None else max(ws_bytes, least)
    ws = torch.empty(max(nb, 1), dtype=torch.uint8, device=DEV)
    size, dev = T.toc_ingest_plan(dblob, off, infos, n_cols, ws)
    buf = torch.zeros(size, dtype=torch.uint8, device=DEV)
    T.toc_ingest_build(dev, dblob, off, buf, ws)
    torch.cuda.synchronize()
    return dev, buf, size


def _host(encs):
    size = T.toc_upload_size(encs)
    buf = torch.zeros(size, dtype=torch.uint8, device=DEV)
    dev = T.toc_upload(encs, buf)
    torch.cuda.synchronize()
    return dev, buf, size


def _ops(dev, W, G):
    info = T.toc_dev_info_get(dev)
    k = W.shape[1]
    Wd, Gd = torch.from_numpy(W).to(DEV), torch.from_numpy(G).to(DEV)
    R = torch.full((info["n_rows"], k), float("nan"), device=DEV)
    out = torch.full((info["n_batches"] * info["n_cols"], k), float("nan"), device=DEV)
    wr, _ = T.toc_workspace_size(dev, T.TOC_OP_RIGHT, k)
    wl, _ = T.toc_workspace_size(dev, T.TOC_OP_LEFT, k)
    ws_r = torch.empty(max(wr // 4, 1), device=DEV) if wr else None
    ws_l = torch.empty(max(wl // 4, 1), device=DEV) if wl else None
    T.toc_right_mul(dev, Wd, R, ws_r)
    T.toc_left_mul(dev, Gd, out, False, ws_l)
    rp = torch.empty(info["n_rows"] + 1, dtype=torch.int64, device=DEV)
    cc = torch.empty(max(info["nnz"], 1), dtype=torch.int32, device=DEV)[:info["nnz"]]
    vv = torch.empty(max(info["nnz"], 1), dtype=torch.float32, device=DEV)[:info["nnz"]]
    T.toc_decode_csr(dev, rp, cc, vv)
    torch.cuda.synchronize()
    return (R.cpu().numpy(), out.cpu().numpy(), rp.cpu().numpy(), cc.cpu().numpy(),
            vv.cpu().numpy().view(np.uint32))


def _check(B, k, ws_bytes=None, seed=0):
    encs = T.toc_encode_batches(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    dh, bh, sh = _host(encs)
    di, bi, si = _ingest(encs, B.n_cols, ws_bytes)
    assert si == sh
    assert T.toc_dev_info_get(di) == T.toc_dev_info_get(dh)
    assert T.toc_dev_layout_get(di) == T.toc_dev_layout_get(dh)
    diff = torch.nonzero(bh != bi).flatten()
    if diff.numel():
        lay = sorted(T.toc_dev_layout_get(dh).items(), key=lambda kv: kv[1])
        at = int(diff[0])
        arr = [n for n, o in lay if o <= at][-1]
        pytest.fail(f"{diff.numel()} image bytes differ; first at {at}, in {arr}")
    rng = np.random.default_rng(seed)
    W = rng.standard_normal((B.n_cols, k)).astype(np.float32)
    G = rng.standard_normal((int(B.n_rows.sum()), k)).astype(np.float32)
    got = _ops(di, W, G)
    want = _ops(dh, W, G)
    for g, w, name in zip(got, want, ("right", "left", "rowptr", "col", "val")):
        assert np.array_equal(g.view(np.uint32) if g.dtype == np.float32 else g,
                              w.view(np.uint32) if w.dtype == np.float32 else w), name
    R, out, rp, cc, vv = got
    flat = []
    for b in range(B.n_batches):
        n, brp, bc, bv = B.batch(b)
        rows = O.canonicalize(n, B.n_cols, brp, bc, bv)
        flat.extend(rows)
        r0 = int(B.row_off[b])
        Rr, S = O.dense_right(rows, B.n_cols, W.astype(np.float64))
        assert np.all(np.abs(R[r0:r0 + n] - Rr) <= TOL * S), f"right, batch {b}"
        Or, S = O.dense_left(rows, B.n_cols, G[r0:r0 + n].astype(np.float64))
        blk = out[b * B.n_cols:(b + 1) * B.n_cols]
        assert np.all(np.abs(blk - Or) <= TOL * S), f"left, batch {b}"
    orp, oc, ov = O.decoded_to_csr(flat)
    assert np.array_equal(rp, orp) and np.array_equal(cc, oc)
    assert np.array_equal(vv, np.asarray(ov, np.float32).view(np.uint32))
    return encs


@pytest.mark.parametrize("cfg,first,nb,k", [
    ("c1", 0, 1, 1), ("c2", 5, 3, 1), ("c3", 11, 4, 300), ("c4", 2, 2, 200), ("c5", 40, 24, 1),
])
def test_config_batches(cfg, first, nb, k):
    _check(config_batches(cfg, first, nb), k)


def test_edge_batches():
    """Empty batches, empty tuples, one-entry tuples and deep prefix trees in one
    upload."""
    parts = [
        Batches(6, [0], np.zeros(1, np.int64), np.zeros(0, np.int32), np.zeros(0, np.float32)),
        Batches(6, [3], np.array([0, 0, 0, 0], np.int64), np.zeros(0, np.int32),
                np.zeros(0, np.float32)),
        Batches(6, [4], np.array([0, 0, 2, 2, 3], np.int64), np.array([1, 3, 1], np.int32),
                np.array([1.5, 2.0, 1.5], np.float32)),
    ]
    for s in range(3):
        rp, c, v = tiny_batch(s, 40, 6, density=0.9, n_values=2, prefix_copy=0.8)
        parts.append(Batches(6, [40], rp, c, v))
    _check(Batches.concat(parts), 5)


def test_small_workspace_many_ranges():
    """A workspace of about three batches' need: the batches go through it in many
    ranges, each range's C' rebuilt in the same scratch."""
    B = config_batches("c3", 100, 12)
    encs = T.toc_encode_batches(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    _, _, infos = _blobs(encs)
    _, least = T.toc_ingest_workspace_size(infos, B.n_cols)
    _check(B, 64, ws_bytes=3 * least)


def test_planned_image_refuses_ops_and_changed_bytes():
    B = config_batches("c5", 0, 4)
    encs = T.toc_encode_batches(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    dblob, off, infos = _blobs(encs)
    full, _ = T.toc_ingest_workspace_size(infos, B.n_cols)
    ws = torch.empty(full, dtype=torch.uint8, device=DEV)
    size, dev = T.toc_ingest_plan(dblob, off, infos, B.n_cols, ws)
    R = torch.empty((int(B.n_rows.sum()), 1), device=DEV)
    W = torch.ones((B.n_cols, 1), device=DEV)
    with pytest.raises(T.TocError):
        T.toc_right_mul(dev, W, R, None)
    # other batches' bytes in place of the planned ones: the build finds that their
    # trees differ from the plan's counts and names the batch; dev stays unbuilt
    B2 = config_batches("c5", 7, 4)
    encs2 = T.toc_encode_batches(B2.n_rows, B2.n_cols, B2.rowptr, B2.col, B2.val)
    dblob2, off2, _ = _blobs(encs2)
    buf = torch.zeros(size, dtype=torch.uint8, device=DEV)
    with pytest.raises(T.TocError, match="batch 0"):
        T.toc_ingest_build(dev, dblob2, off2, buf, ws)
    with pytest.raises(T.TocError):
        T.toc_right_mul(dev, W, R, None)
    buf = torch.zeros(size, dtype=torch.uint8, device=DEV)
    with pytest.raises(T.TocError):
        T.toc_ingest_build(dev, dblob, off, buf[:size - 1], ws)
    T.toc_ingest_build(dev, dblob, off, buf, ws)
    wr, _ = T.toc_workspace_size(dev, T.TOC_OP_RIGHT, 1)
    T.toc_right_mul(dev, W, R, torch.empty(max(wr // 4, 1), device=DEV) if wr else None)
    torch.cuda.synchronize()
    assert torch.isfinite(R).all().item()


def test_malformed_blob_named():
    """A code naming a node that does not exist yet: the plan fails and names the
    batch (the status toc_cprime_build gives it)."""
    B = config_batches("c5", 0, 3)
    encs = T.toc_encode_batches(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    blobs = [np.array(T.toc_enc_pack(e)) for e in encs]
    infos = [T.toc_phys_info_get(b) for b in blobs]
    bad = blobs[1]
    # D's array is the fourth; its first code names node 1 at least, so a code one
    # past the nodes existing at that point is malformed
    pos = 0
    for a in range(3):
        cnt = int.from_bytes(bytes(bad[pos:pos + 4]), "little")
        pos += 5 + cnt * int(bad[pos + 4])
    w = int(bad[pos + 4])
    first = pos + 5
    big = infos[1]["n_nodes"] + 5
    bad[first:first + w] = np.frombuffer(int(min(big, 256 ** w - 1)).to_bytes(w, "little"), np.uint8)
    off = np.concatenate([[0], np.cumsum([len(b) for b in blobs])]).astype(np.int64)
    dblob = torch.from_numpy(np.concatenate(blobs + [np.zeros(1, np.uint8)])).to(DEV)
    full, _ = T.toc_ingest_workspace_size(infos, B.n_cols)
    ws = torch.empty(full, dtype=torch.uint8, device=DEV)
    with pytest.raises(T.TocError, match="batch 1"):
        T.toc_ingest_plan(dblob, off, infos, B.n_cols, ws)
