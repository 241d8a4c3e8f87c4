"""GPU parity of the products' summation: blocked sums keep every serial chain of
fp32 additions short, so |gpu - oracle| <= 1e-5 * S holds by construction and not
by luck (Theorems 1 and 2 are exact only in exact arithmetic).

* Many work items per persistent worker on the dense quantised workload (250 x
  1,000 batches, k = 200): the right product takes the staged kernel (the deep H
  rows of a batch do not fit in LDS) and each worker takes several (batch, column
  tile) items in turn, reloading its W tile and reusing its workspace slot.
* Adversarial sums: one large term followed by hundreds of terms a quarter of an
  ulp of it.  Summed serially in binary32 every small term is lost and the error
  exceeds 1e-5 * S (checked on the CPU below); summed in blocks it stays far
  inside.  Each case is built to run through one kernel of the path.
"""

import multiprocessing as mp

import numpy as np
import pytest

import oracle as O
import paper_1702_06943_amd as T
from workloads import Batches, config_batches, config_G, config_W
from workloads.parallel import default_workers

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TOL = 1e-5
TINY = np.float32(2.0 ** -25)       # a quarter of an ulp of 1.0


def _upload(B, flags=0):
    encs = T.toc_encode_batches(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    buf = torch.empty(T.toc_upload_size(encs, flags), dtype=torch.uint8, device=DEV)
    dev = T.toc_upload(encs, buf, flags)
    return dev, buf, T.toc_dev_info_get(dev)


def _right(dev, info, W):
    k = W.shape[1]
    Wd = torch.from_numpy(np.ascontiguousarray(W)).to(DEV)
    R = torch.full((info["n_rows"], k), float("nan"), device=DEV)
    ws_n, _ = T.toc_workspace_size(dev, T.TOC_OP_RIGHT, k)
    ws = torch.empty(max(ws_n, 4) // 4, device=DEV) if ws_n else None
    T.toc_right_mul(dev, Wd, R, ws)
    torch.cuda.synchronize()
    return R.cpu().numpy().astype(np.float64)


def _left(dev, info, G):
    k = G.shape[1]
    Gd = torch.from_numpy(np.ascontiguousarray(G)).to(DEV)
    out = torch.full((info["n_batches"] * info["n_cols"], k), float("nan"), device=DEV)
    ws_n, _ = T.toc_workspace_size(dev, T.TOC_OP_LEFT, k)
    ws = torch.empty(max(ws_n, 4) // 4, device=DEV) if ws_n else None
    T.toc_left_mul(dev, Gd, out, False, ws)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64)


def _serial_f32(terms):
    """The terms summed one after another in binary32 (what one accumulator does)."""
    s = np.float32(0.0)
    for t in np.asarray(terms, np.float32):
        s = np.float32(s + t)
    return float(s)


def _assert_adversarial(terms):
    """A serial binary32 sum of these terms (in this order) breaks the tolerance."""
    exact = float(np.sum(np.asarray(terms, np.float64)))
    S = float(np.sum(np.abs(np.asarray(terms, np.float64))))
    assert abs(_serial_f32(terms) - exact) > TOL * S


def _check(got, ref, S, what):
    err = np.abs(got - ref)
    ratio = float(np.max(err / np.maximum(S, 1e-300)))
    assert np.all(err <= TOL * S), f"{what}: max err/S {ratio:.3e}"
    return ratio


def _pool():
    ctx = "spawn" if torch.cuda.is_initialized() else "fork"
    return mp.get_context(ctx).Pool(min(default_workers(), 16))


@pytest.mark.timeout(600)
def test_dense_quantised_many_items_per_worker():
    """96 batches of the dense quantised workload at k = 200: 7 column tiles per
    batch, 84 items on each XCD's 32 workers, so every worker runs several items
    (right: staged kernel, W tile reloaded between items, workspace slot reused;
    left: tiled kernel with tree rows partly in the workspace).  Every batch is
    compared element by element with the oracle; decode bit for bit."""
    import oracle_jobs
    cfg, nb, k = "c4", 96, 200
    B = config_batches(cfg, 0, nb)
    W = config_W(cfg, k)
    G = config_G(cfg, 0, nb, k)
    dev, buf, info = _upload(B)
    R = _right(dev, info, W)
    out = _left(dev, info, G)
    rp = torch.empty(info["n_rows"] + 1, dtype=torch.int64, device=DEV)
    cc = torch.empty(info["nnz"], dtype=torch.int32, device=DEV)
    vv = torch.empty(info["nnz"], dtype=torch.float32, device=DEV)
    T.toc_decode_csr(dev, rp, cc, vv)
    torch.cuda.synchronize()
    rp, cc, vv = rp.cpu().numpy(), cc.cpu().numpy(), vv.cpu().numpy().view(np.uint32)
    print(f"{nb} batches uploaded ({info['n_deep']} deep codes); oracle on a pool", flush=True)
    pool = _pool()
    try:
        refs = pool.map(oracle_jobs.products, [(cfg, b, W, k) for b in range(nb)])
    finally:
        pool.close()
        pool.join()
    m, n = B.n_cols, 250
    worst = 0.0
    for b, (Rr, SR, Or, SO, crp, ccol, cval) in enumerate(refs):
        worst = max(worst, _check(R[b * n:(b + 1) * n], Rr, SR, f"right, batch {b}"))
        worst = max(worst, _check(out[b * m:(b + 1) * m], Or, SO, f"left, batch {b}"))
        p0, p1 = int(rp[b * n]), int(rp[(b + 1) * n])
        assert np.array_equal(rp[b * n:(b + 1) * n + 1] - p0, crp), f"decode rowptr, batch {b}"
        assert np.array_equal(cc[p0:p1], ccol), f"decode col, batch {b}"
        assert np.array_equal(vv[p0:p1], cval), f"decode val, batch {b}"
    print(f"max |err|/S over {nb} batches: {worst:.3e}", flush=True)


def _batch(rows, n_cols):
    """rows: list of (cols, vals) -> one-batch Batches."""
    rp = np.cumsum([0] + [len(c) for c, _ in rows]).astype(np.int64)
    col = np.concatenate([np.asarray(c, np.int32) for c, _ in rows]) if rows else \
        np.zeros(0, np.int32)
    val = np.concatenate([np.asarray(v, np.float32) for _, v in rows]) if rows else \
        np.zeros(0, np.float32)
    return Batches(n_cols, [len(rows)], rp, col, val)


def _long_row(n_cols):
    """1.0 at column 0, then TINY in every other column."""
    v = np.full(n_cols, TINY, np.float32)
    v[0] = 1.0
    return np.arange(n_cols, dtype=np.int32), v


def _right_case(B, k, rows_of_interest=None):
    dev, buf, info = _upload(B)
    W = np.ones((B.n_cols, k), np.float32)
    R = _right(dev, info, W)
    worst = 0.0
    for b in range(B.n_batches):
        n, rp, c, v = B.batch(b)
        rows = O.canonicalize(n, B.n_cols, rp, c, v)
        Rr, S = O.dense_right(rows, B.n_cols, W)
        r0 = int(B.row_off[b])
        worst = max(worst, _check(R[r0:r0 + n], Rr, S, f"right, batch {b}"))
    return worst


def test_blocked_right_tiled_long_tuple():
    """A tuple of 1,200 depth-1 codes through the tiled right product (k = 32)."""
    m = 1200
    c, v = _long_row(m)
    _assert_adversarial(v)
    B = _batch([(c, v), ([3, 7], [0.5, -2.0])], m)
    _right_case(B, 32)


def test_blocked_right_staged_long_tuple():
    """The same tuple shape (1,000 codes) through the staged right product: the
    batch is uploaded with a dense quantised batch, whose deep H rows do not fit
    in LDS, so every batch of the upload takes the staged kernel (k = 40: a full
    and a partial column tile)."""
    c4 = config_batches("c4", 3, 1)
    c, v = _long_row(c4.n_cols)
    _assert_adversarial(v)
    B = Batches.concat([c4, _batch([(c, v)], c4.n_cols)])
    _right_case(B, 40)


def test_blocked_right_wide_long_tuple():
    """2,000 codes with k = 8: the W tile does not fit in LDS (wide kernel)."""
    m = 2000
    c, v = _long_row(m)
    _assert_adversarial(v)
    _right_case(_batch([(c, v)], m), 8)


def test_blocked_right_k1_long_tuple():
    """k = 1: one tuple of 4,800 codes among 200 one-code tuples (so that few
    lanes sum a tuple: each lane's share of the long tuple is 1,200 codes)."""
    m = 4800
    c, v = _long_row(m)
    _assert_adversarial(v[::4])         # lane 0's share, in its order
    rows = [(c, v)] + [([i % m], [1.0 + i]) for i in range(200)]
    _right_case(_batch(rows, m), 1)


def _column_batch(n_rows, n_cols=4):
    """Column 0 of a batch: 1.0 in tuple 0, then n_rows - 1 tuples each holding
    its own value v_i (all distinct, so every pair is its own depth-1 leaf) whose
    G row is TINY / v_i: every term of the column after the first is about TINY.
    Returns the batch and G (k columns filled alike by the caller)."""
    vals = (1.0 + np.arange(1, n_rows) * 2.0 ** -12).astype(np.float32)
    rows = [([0], [1.0])] + [([0], [x]) for x in vals]
    g = np.concatenate([[1.0], (TINY / vals.astype(np.float64))]).astype(np.float32)
    terms = np.concatenate([[1.0], vals.astype(np.float64) * g[1:]])
    _assert_adversarial(terms)
    return _batch(rows, n_cols), g


@pytest.mark.parametrize("n_rows,k", [(600, 64), (1000, 64), (600, 1), (3000, 1), (1500, 4)])
def test_blocked_left_long_column(n_rows, k):
    """A key column with n_rows leaf occurrences: 600 rows take the 64-column
    tiled left product, 1,000 rows the 32-column one (8-lane groups), 1,500 rows
    at k = 4 the wide kernel, k = 1 the LDS-resident kernel."""
    B, g = _column_batch(n_rows)
    G = np.repeat(g[:, None], k, axis=1)
    dev, buf, info = _upload(B)
    out = _left(dev, info, G)
    n, rp, c, v = B.batch(0)
    rows = O.canonicalize(n, B.n_cols, rp, c, v)
    ref, S = O.dense_left(rows, B.n_cols, G)
    _check(out, ref, S, "left")
