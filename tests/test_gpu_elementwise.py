"""GPU parity of the element-wise operations against the oracle.

toc_map_values (Algorithm 3: A.*c and A.^2 by changing the key values) must give,
bit for bit, the oracle's decode of the modified I, and the products computed
afterwards must match the oracle's dense products of the modified batch within
1e-5 * S.  toc_decode_dense (Algorithm 9: dense A .+ c) must match the oracle's
dense matrix bit for bit, leaving the padding columns of A untouched.
"""

import numpy as np
import pytest

import oracle as O
import paper_1702_06943_amd as T
from workloads import config_batches, config_G, config_W

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TOL = 1e-5


def _upload(B, flags=0):
    encs = T.toc_encode_batches(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    buf = torch.empty(T.toc_upload_size(encs, flags), dtype=torch.uint8, device=DEV)
    return encs, buf, T.toc_upload(encs, buf, flags)


def _oracle_rows(B, b, op=None, c=0.0):
    n, rp, col, val = B.batch(b)
    rows = O.canonicalize(n, B.n_cols, rp, col, val)
    if op is None:
        return rows
    I, D, _ = O.encode(rows)
    return O.decode(O.map_values(I, op, c), D)


def _decode(dev, info):
    rp = torch.full((info["n_rows"] + 1,), -7, dtype=torch.int64, device=DEV)
    cd = torch.full((info["nnz"],), -7, dtype=torch.int32, device=DEV)
    vd = torch.full((info["nnz"],), float("nan"), dtype=torch.float32, device=DEV)
    T.toc_decode_csr(dev, rp, cd, vd)
    torch.cuda.synchronize()
    return rp.cpu().numpy(), cd.cpu().numpy(), vd.cpu().numpy()


@pytest.mark.parametrize("cfg,nb,k", [("c1", 1, 3), ("c3", 2, 40), ("c4", 1, 200),
                                      ("c5", 4, 1), ("c2", 2, 1)])
@pytest.mark.parametrize("op,c", [(0, 0.37), (1, 0.0), (0, -2.0)])
@pytest.mark.parametrize("flags", [0, T.TOC_UPLOAD_KEEP_DEAD])
def test_map_values(cfg, nb, k, op, c, flags):
    print(f"map_values {cfg} nb={nb} k={k} op={op} c={c} flags={flags}", flush=True)
    B = config_batches(cfg, 3, nb)
    encs, buf, dev = _upload(B, flags)
    info = T.toc_dev_info_get(dev)
    T.toc_map_values(dev, op, c)
    rows = [_oracle_rows(B, b, op, c) for b in range(nb)]
    # decode: bit-exact
    rp_o, c_o, v_o = O.decoded_to_csr([r for rs in rows for r in rs])
    rp_g, c_g, v_g = _decode(dev, info)
    assert np.array_equal(rp_g, rp_o) and np.array_equal(c_g, c_o)
    assert np.array_equal(v_g.view(np.uint32), v_o.view(np.uint32))
    # products of the modified batch
    W = config_W(cfg, k)
    G = config_G(cfg, 3, nb, k)
    R = torch.full((info["n_rows"], k), float("nan"), device=DEV)
    ws_n, _ = T.toc_workspace_size(dev, T.TOC_OP_RIGHT, k)
    ws = torch.empty(max(ws_n, 4) // 4, device=DEV) if ws_n else None
    T.toc_right_mul(dev, torch.from_numpy(W).to(DEV), R, ws)
    out = torch.full((nb * B.n_cols, k), float("nan"), device=DEV)
    ws_n, _ = T.toc_workspace_size(dev, T.TOC_OP_LEFT, k)
    ws = torch.empty(max(ws_n, 4) // 4, device=DEV) if ws_n else None
    T.toc_left_mul(dev, torch.from_numpy(G).to(DEV), out, False, ws)
    torch.cuda.synchronize()
    R, out = R.cpu().numpy().astype(np.float64), out.cpu().numpy().astype(np.float64)
    m = B.n_cols
    for b in range(nb):
        r0, n = int(B.row_off[b]), int(B.row_off[b + 1] - B.row_off[b])
        R_ref, S = O.dense_right(rows[b], m, W)
        assert np.all(np.abs(R[r0:r0 + n] - R_ref) <= TOL * S)
        o_ref, S = O.dense_left(rows[b], m, G[r0:r0 + n])
        assert np.all(np.abs(out[b * m:(b + 1) * m] - o_ref) <= TOL * S)


def test_map_values_twice_and_identity():
    B = config_batches("c3", 0, 2)
    encs, buf, dev = _upload(B)
    info = T.toc_dev_info_get(dev)
    before = _decode(dev, info)
    T.toc_map_values(dev, T.TOC_MAP_SCALE, 1.0)
    assert all(np.array_equal(x, y) for x, y in zip(before, _decode(dev, info)))
    # scaling by 2 then by 0.5 is exact for these values
    T.toc_map_values(dev, T.TOC_MAP_SCALE, 2.0)
    T.toc_map_values(dev, T.TOC_MAP_SCALE, 0.5)
    after = _decode(dev, info)
    assert np.array_equal(after[2].view(np.uint32), before[2].view(np.uint32))


@pytest.mark.parametrize("cfg,nb", [("c1", 1), ("c3", 3), ("c4", 1), ("c5", 8), ("c2", 2)])
@pytest.mark.parametrize("c", [0.0, -1.25])
def test_decode_dense(cfg, nb, c):
    print(f"decode_dense {cfg} nb={nb} c={c}", flush=True)
    B = config_batches(cfg, 1, nb)
    encs, buf, dev = _upload(B)
    info = T.toc_dev_info_get(dev)
    m, pad = B.n_cols, 5
    A = torch.full((info["n_rows"], m + pad), float("nan"), device=DEV)
    T.toc_decode_dense(dev, A[:, :m], c)
    torch.cuda.synchronize()
    A = A.cpu().numpy()
    want = np.concatenate([O.dense_plus(_oracle_rows(B, b), m, c) for b in range(nb)])
    assert np.array_equal(A[:, :m].view(np.uint32), want.view(np.uint32))
    assert np.all(np.isnan(A[:, m:]))


def test_decode_dense_after_map():
    B = config_batches("c4", 2, 1)
    encs, buf, dev = _upload(B)
    info = T.toc_dev_info_get(dev)
    T.toc_map_values(dev, T.TOC_MAP_SQUARE)
    A = torch.empty((info["n_rows"], B.n_cols), device=DEV)
    T.toc_decode_dense(dev, A, 0.5)
    torch.cuda.synchronize()
    want = O.dense_plus(_oracle_rows(B, 0, O.MAP_SQUARE), B.n_cols, 0.5)
    assert np.array_equal(A.cpu().numpy().view(np.uint32), want.view(np.uint32))


def test_elementwise_errors():
    B = config_batches("c1", 0, 1)
    encs, buf, dev = _upload(B)
    with pytest.raises(T.TocError) as ei:
        T.toc_map_values(dev, 7, 1.0)
    assert ei.value.status == T.TOC_EINVAL
    with pytest.raises(T.TocError) as ei:
        T.toc_map_values(dev, T.TOC_MAP_SCALE, float("inf"))
    assert ei.value.status == T.TOC_EINVAL
    A = torch.empty((250, 68), device=DEV)
    with pytest.raises(T.TocError):
        T.toc_decode_dense(dev, A, float("nan"))
    lib = T.lib()
    assert lib.toc_decode_dense(dev.handle, 0.0, A.data_ptr(), 67, None) == T.TOC_EINVAL
