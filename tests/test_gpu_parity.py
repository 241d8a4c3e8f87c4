"""GPU parity: the HIP path (through the C ABI) against the oracle.

Decode must be bit-exact; products must satisfy |gpu - oracle| <= 1e-5 * S per
element, where S is the sum of absolute values of the terms (S = 0 -> exactly 0).
"""

import json
import os

import numpy as np
import pytest

import oracle as O
import paper_1702_06943_amd as T
from workloads import config_batches, config_G, config_W, tiny_batch, Batches

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
GOLD = json.load(open(os.path.join(HERE, "golden", "worked_example.json")))
TOL = 1e-5
DEV = "cuda:0"


def _batches_from_csrs(csrs, n_cols):
    """list of (n_rows, rowptr, col, val) -> Batches"""
    parts = []
    for n, rp, c, v in csrs:
        parts.append(Batches(n_cols, [n], rp, c, v))
    return Batches.concat(parts)


def run_gpu(B, W=None, G=None, flags=0, ws_scale=None, accumulate_init=None,
            ld_pad=0, decode=True):
    """Encode, upload and run right, left and decode.  Returns host arrays."""
    encs = T.toc_encode_batches(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    size = T.toc_upload_size(encs, flags)
    buf = torch.empty(size, dtype=torch.uint8, device=DEV)
    dev = T.toc_upload(encs, buf, flags)
    info = T.toc_dev_info_get(dev)
    res = {"info": info}
    if W is not None:
        k = W.shape[1]
        Wd = torch.zeros((W.shape[0], k + ld_pad), device=DEV)
        Wd[:, :k] = torch.from_numpy(W)
        Wv = Wd[:, :k]
        Rd = torch.full((info["n_rows"], k + ld_pad), float("nan"), device=DEV)[:, :k]
        ws_n, ws_min = T.toc_workspace_size(dev, T.TOC_OP_RIGHT, k)
        if ws_scale is not None and ws_n:
            ws_n = max(ws_min, int(ws_min * ws_scale))
        ws = torch.empty(max(ws_n, 4) // 4, device=DEV) if ws_n else None
        T.toc_right_mul(dev, Wv, Rd, ws)
        torch.cuda.synchronize()
        res["R"] = Rd.cpu().numpy()
    if G is not None:
        k = G.shape[1]
        Gd = torch.zeros((G.shape[0], k + ld_pad), device=DEV)
        Gd[:, :k] = torch.from_numpy(G)
        Gv = Gd[:, :k]
        rows_out = info["n_batches"] * info["n_cols"]
        if accumulate_init is not None:
            Od = torch.from_numpy(accumulate_init).to(DEV)
        else:
            Od = torch.full((rows_out, k + ld_pad), float("nan"), device=DEV)[:, :k]
        ws_n, ws_min = T.toc_workspace_size(dev, T.TOC_OP_LEFT, k)
        if ws_scale is not None and ws_n:
            ws_n = max(ws_min, int(ws_min * ws_scale))
        ws = torch.empty(max(ws_n, 4) // 4, device=DEV) if ws_n else None
        T.toc_left_mul(dev, Gv, Od, accumulate_init is not None, ws)
        torch.cuda.synchronize()
        res["out"] = Od.cpu().numpy()
    if decode:
        rp = torch.full((info["n_rows"] + 1,), -7, dtype=torch.int64, device=DEV)
        cd = torch.full((info["nnz"],), -7, dtype=torch.int32, device=DEV)
        vd = torch.full((info["nnz"],), float("nan"), dtype=torch.float32, device=DEV)
        T.toc_decode_csr(dev, rp, cd, vd)
        torch.cuda.synchronize()
        res["csr"] = (rp.cpu().numpy(), cd.cpu().numpy(), vd.cpu().numpy())
    return res


def check_against_oracle(B, res, W=None, G=None, batches=None, accumulate_init=None):
    """Per-batch comparison; returns the max |err|/S seen."""
    worst = 0.0
    r0 = 0
    all_rows = []
    for b in range(B.n_batches) if batches is None else batches:
        n, rp, c, v = B.batch(b)
        rows = O.canonicalize(n, B.n_cols, rp, c, v)
        r0 = int(B.row_off[b])
        if W is not None:
            R_ref, S = O.dense_right(rows, B.n_cols, W)
            got = res["R"][r0:r0 + n].astype(np.float64)
            err = np.abs(got - R_ref)
            assert np.all(err <= TOL * S), f"right mul batch {b}: max err/S " \
                f"{np.max(err / np.maximum(S, 1e-300))}"
            worst = max(worst, float(np.max(err / np.maximum(S, 1e-300), initial=0)))
        if G is not None:
            g = G[r0:r0 + n]
            out_ref, S = O.dense_left(rows, B.n_cols, g)
            m = B.n_cols
            got = res["out"][b * m:(b + 1) * m].astype(np.float64)
            if accumulate_init is not None:
                got = got - accumulate_init[b * m:(b + 1) * m].astype(np.float64)
                S = S + np.abs(accumulate_init[b * m:(b + 1) * m]) * 1e-2
            err = np.abs(got - out_ref)
            assert np.all(err <= TOL * S), f"left mul batch {b}: max err/S " \
                f"{np.max(err / np.maximum(S, 1e-300))}"
            worst = max(worst, float(np.max(err / np.maximum(S, 1e-300), initial=0)))
        all_rows.append(rows)
    if "csr" in res and batches is None:
        rp_g, c_g, v_g = res["csr"]
        flat = [r for rows in all_rows for r in rows]
        rp_o, c_o, v_o = O.decoded_to_csr(flat)
        assert np.array_equal(rp_g, rp_o)
        assert np.array_equal(c_g, c_o)
        assert np.array_equal(v_g.view(np.uint32), v_o.view(np.uint32))
    return worst


def test_worked_example():
    rows_in = GOLD["rows_from_table2"]["rows"]
    rp = np.cumsum([0] + [len(r) for r in rows_in])
    c = np.array([p[0] for r in rows_in for p in r], np.int32)
    v = np.array([p[1] for r in rows_in for p in r], np.float32)
    B = Batches(4, [4], rp, c, v)
    ones = np.ones((4, 1), np.float32)
    res = run_gpu(B, W=ones, G=ones)
    assert np.allclose(res["R"][:, 0], GOLD["products_all_ones"]["right"], atol=1e-6)
    assert np.allclose(res["out"][:, 0], GOLD["products_all_ones"]["left"], atol=1e-6)
    check_against_oracle(B, res, W=ones, G=ones)


TINY = [
    dict(n_rows=12, density=0.9, n_values=2, prefix_copy=0.8),
    dict(n_rows=30, density=0.5, n_values=3, prefix_copy=0.5),
    dict(n_rows=3, density=0.0, n_values=1),                 # all-zero batch
    dict(n_rows=1, density=1.0, n_values=1),                 # one dense row
    dict(n_rows=0, density=0.5, n_values=2),                 # empty batch
    dict(n_rows=70, density=0.3, n_values=4, prefix_copy=0.3),
    dict(n_rows=9, density=0.05, n_values=2),                # mostly empty rows
]


def _tiny_set(seed, n_cols=40, zeros=True):
    csrs = []
    for i, spec in enumerate(TINY):
        rp, c, v = tiny_batch(900 + seed * 13 + i, n_cols=n_cols, zeros=zeros, **spec)
        csrs.append((spec["n_rows"], rp, c, v))
    return _batches_from_csrs(csrs, n_cols)


@pytest.mark.parametrize("k", [1, 3, 64, 65, 300, 513])
@pytest.mark.parametrize("flags", [0, T.TOC_UPLOAD_KEEP_DEAD])
def test_tiny_batches(k, flags):
    B = _tiny_set(k + flags)
    rng = np.random.default_rng(k)
    W = rng.standard_normal((B.n_cols, k)).astype(np.float32)
    G = rng.standard_normal((int(B.n_rows.sum()), k)).astype(np.float32)
    res = run_gpu(B, W=W, G=G, flags=flags)
    check_against_oracle(B, res, W=W, G=G)


def test_integer_inputs_exact():
    """Small integers: every partial sum is exact in fp32, so results are exact."""
    csrs = []
    for i in range(5):
        rp, c, v = tiny_batch(40 + i, n_rows=40, n_cols=30, density=0.7, n_values=3,
                              integer=True, prefix_copy=0.7)
        csrs.append((40, rp, c, v))
    B = _batches_from_csrs(csrs, 30)
    rng = np.random.default_rng(3)
    for k in (1, 70):
        W = rng.integers(-3, 4, size=(30, k)).astype(np.float32)
        G = rng.integers(-3, 4, size=(200, k)).astype(np.float32)
        res = run_gpu(B, W=W, G=G, decode=False)
        for b in range(5):
            n, rp, c, v = B.batch(b)
            A = np.zeros((n, 30))
            for i in range(n):
                A[i, c[rp[i]:rp[i + 1]]] = v[rp[i]:rp[i + 1]]
            assert np.array_equal(res["R"][b * 40:(b + 1) * 40], A @ W)
            assert np.array_equal(res["out"][b * 30:(b + 1) * 30], A.T @ G[b * 40:(b + 1) * 40])


@pytest.mark.parametrize("cfg,nb,k", [("c1", 1, 1), ("c2", 3, 1), ("c3", 3, 300),
                                      ("c4", 1, 200), ("c5", 8, 1), ("c3", 2, 1),
                                      ("c2", 2, 16), ("c5", 4, 33)])
def test_config_batches(cfg, nb, k):
    B = config_batches(cfg, 5 if cfg != "c1" else 0, nb)
    W = config_W(cfg, k)
    G = config_G(cfg, 5 if cfg != "c1" else 0, nb, k)
    res = run_gpu(B, W=W, G=G)
    worst = check_against_oracle(B, res, W=W, G=G)
    print(f"{cfg} nb={nb} k={k}: max err/S = {worst:.3e}")


def test_right_batch_pairs():
    """27 batches of the c3 shape: the tiled right product takes the batches of an
    XCD (b, b + 8, ...) two per work item when both batches' deep H rows fit in
    LDS beside the W tile, and the last batch of an XCD with an odd count alone."""
    B = config_batches("c3", 11, 27)
    k = 40
    W = config_W("c3", k)
    res = run_gpu(B, W=W, decode=False)
    check_against_oracle(B, res, W=W)


def _host_deep(B):
    """Deep (depth >= 2) codes of each batch, from a host image of that batch."""
    out = []
    for b in range(B.n_batches):
        n, rp, c, v = B.batch(b)
        one = _batches_from_csrs([(n, rp, c, v)], B.n_cols)
        encs = T.toc_encode_batches(one.n_rows, one.n_cols, one.rowptr, one.col, one.val)
        buf = np.zeros(T.toc_upload_size(encs, T.TOC_UPLOAD_HOST), np.uint8)
        out.append(T.toc_dev_info_get(T.toc_upload(encs, buf, T.TOC_UPLOAD_HOST))["n_deep"])
    return out


def test_right_pairs_that_do_not_fit():
    """n_cols = 1100: a 32-column W tile leaves LDS room for 178 deep H rows.
    Every batch fits alone and some pairs (b, b + 8) do not, so the tiled right
    product takes one batch per work item."""
    n_cols = 1100
    csrs = []
    for i in range(24):
        rp, c, v = tiny_batch(300 + i, n_rows=40, n_cols=n_cols, density=0.04, n_values=3,
                              prefix_copy=0.2)
        csrs.append((40, rp, c, v))
    B = _batches_from_csrs(csrs, n_cols)
    deep = _host_deep(B)
    room = (160 * 1024 - 16 - (n_cols + 1) * 128) // 128
    assert max(deep) <= room
    assert max(deep[b] + deep[b + 8] for b in range(16) if (b // 8) % 2 == 0) > room
    k = 45
    W = np.random.default_rng(4).standard_normal((n_cols, k)).astype(np.float32)
    res = run_gpu(B, W=W, decode=False)
    check_against_oracle(B, res, W=W)


def test_accumulate_and_strides():
    B = _tiny_set(5)
    rng = np.random.default_rng(11)
    for k in (1, 5, 130):
        W = rng.standard_normal((B.n_cols, k)).astype(np.float32)
        G = rng.standard_normal((int(B.n_rows.sum()), k)).astype(np.float32)
        init = rng.standard_normal((B.n_batches * B.n_cols, k)).astype(np.float32)
        res = run_gpu(B, W=W, G=G, ld_pad=7, accumulate_init=init)
        check_against_oracle(B, res, W=W, G=G, accumulate_init=init)


def test_small_workspace_multiple_passes():
    B = config_batches("c4", 0, 2)
    B2 = _tiny_set(2, n_cols=B.n_cols, zeros=False)
    B = Batches.concat([B, B2])
    k = 40
    rng = np.random.default_rng(5)
    W = rng.standard_normal((B.n_cols, k)).astype(np.float32)
    G = rng.standard_normal((int(B.n_rows.sum()), k)).astype(np.float32)
    res = run_gpu(B, W=W, G=G, ws_scale=1.0)
    check_against_oracle(B, res, W=W, G=G)


def test_huge_single_row_and_large_batch():
    """One row of 20,000 pairs; and a batch whose live codes exceed LDS (k = 1
    falls back to the workspace kernels)."""
    rng = np.random.default_rng(8)
    n_cols = 20000
    v1 = rng.choice(np.array([1.5, -2.0], np.float32), size=n_cols)
    row = (1, np.array([0, n_cols]), np.arange(n_cols, dtype=np.int32), v1)
    rows = 250
    dense = rng.standard_normal((rows, 400)).astype(np.float32)   # all pairs distinct
    rp = np.arange(rows + 1) * 400
    cols = np.tile(np.arange(400, dtype=np.int32), rows)
    big = (rows, rp, cols, dense.ravel())
    B = _batches_from_csrs([row, big], n_cols)
    for k in (1, 2):
        W = rng.standard_normal((n_cols, k)).astype(np.float32)
        G = rng.standard_normal((rows + 1, k)).astype(np.float32)
        res = run_gpu(B, W=W, G=G)
        check_against_oracle(B, res, W=W, G=G)


def _tree_occurrences(B):
    """Per batch: (tree codes, entries of the tree codes' own occurrences), read
    from the host-built image (toc_upload to host memory)."""
    encs = T.toc_encode_batches(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    buf = np.zeros(T.toc_upload_size(encs), np.uint8)
    dev = T.toc_upload(encs, buf, T.TOC_UPLOAD_HOST)
    L = T.toc_dev_layout_get(dev)
    recs = np.frombuffer(buf[L["batches"]:L["batches"] + 96 * B.n_batches].tobytes(), np.uint8)
    out = []
    for b in range(B.n_batches):
        rec = recs[96 * b:96 * (b + 1)].tobytes()
        code_base = int(np.frombuffer(rec[:8], np.int64)[0])
        _, n_codes, n1, ni, _, n_d, _, _ = (int(x) for x in np.frombuffer(rec[64:], np.int32))
        n_tree = ni + n_codes - n1
        off = np.frombuffer(buf[L["occ_off"] + 4 * (code_base + 2 * b):][:4 * (n_codes + 2)]
                            .tobytes(), np.uint32)
        out.append((n_tree, n_d + n_tree - int(off[n1 - ni + 1])))
    return out


def test_left_tree_occurrences_in_and_beyond_lds():
    """The tiled left product copies a batch's tree-code occurrences into LDS when
    they fit in 1,024 words and reads them from memory otherwise: one batch of
    each kind (rows copying long prefixes of earlier rows make many tree codes
    with many occurrences) in one launch, right and left against the oracle."""
    m = 40
    heavy = tiny_batch(7, 480, m, density=0.9, n_values=1, prefix_copy=0.99)
    light = tiny_batch(8, 480, m, density=0.2, n_values=30)
    B = _batches_from_csrs([(480,) + heavy, (480,) + light], m)
    occ = _tree_occurrences(B)
    assert occ[0][1] > 1024 >= occ[1][1], occ
    rng = np.random.default_rng(31)
    for k in (64, 40):
        W = rng.standard_normal((m, k)).astype(np.float32)
        G = rng.standard_normal((960, k)).astype(np.float32)
        res = run_gpu(B, W=W, G=G)
        check_against_oracle(B, res, W=W, G=G)


def test_decode_batch_of_many_runs():
    """A batch of 8,000 short rows over 6 columns: few codes (its keys and links fit
    the batch decode's LDS) but more than eight runs of 1,024 entries of D, so the
    batch decode loads its codes in more than one group of runs."""
    rp, c, v = tiny_batch(21, 8000, 6, density=0.7, n_values=2)
    B = _batches_from_csrs([(8000, rp, c, v)], 6)
    encs = T.toc_encode_batches(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    assert T.toc_enc_info_get(encs[0])["n_codes"] > 8 * 1024
    rng = np.random.default_rng(12)
    W = rng.standard_normal((6, 1)).astype(np.float32)
    G = rng.standard_normal((8000, 1)).astype(np.float32)
    res = run_gpu(B, W=W, G=G)
    check_against_oracle(B, res, W=W, G=G)


def _one_pair_rows(lengths, n_cols, n_values, offset=0):
    """A batch whose rows hold one pair each (or none, where lengths has 0), so
    that its D has exactly one entry per non-empty row; pair i is column
    i % n_cols with value 1 + (i // n_cols) % n_values."""
    lengths = np.asarray(lengths, np.int64)
    rp = np.concatenate([[0], np.cumsum(lengths)])
    i = np.arange(int(rp[-1])) + offset
    c = (i % n_cols).astype(np.int32)
    v = (1 + (i // n_cols) % n_values).astype(np.float32)
    return len(lengths), rp, c, v


def test_decode_runs_of_exact_length():
    """D of 2,048, 8,192 and 8,193 entries (whole runs of 1,024, a whole group of
    eight runs, one entry past it), with empty tuples starting at a run boundary
    and at the end of D, through the batch decode; then 9,216 distinct pairs
    (keys beyond the batch decode's LDS) through the CSR decode."""
    few = [_one_pair_rows([1] * 1024 + [0] * 3 + [1] * 1024 + [0] * 2, 6, 2),
           _one_pair_rows([1] * 8192, 6, 2),
           _one_pair_rows([0] + [1] * 8193, 6, 2)]
    B = _batches_from_csrs(few, 6)
    rng = np.random.default_rng(13)
    W = rng.standard_normal((6, 1)).astype(np.float32)
    G = rng.standard_normal((int(B.n_rows.sum()), 1)).astype(np.float32)
    check_against_oracle(B, run_gpu(B, W=W, G=G), W=W, G=G)
    many = [_one_pair_rows([1] * 4096 + [0] + [1] * 5120 + [0], 96, 96)]
    B = _batches_from_csrs(many, 96)
    encs = T.toc_encode_batches(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    assert 8 * T.toc_enc_info_get(encs[0])["n_live"] > 64 * 1024   # keys beyond 64 KiB
    W = rng.standard_normal((96, 1)).astype(np.float32)
    G = rng.standard_normal((int(B.n_rows.sum()), 1)).astype(np.float32)
    check_against_oracle(B, run_gpu(B, W=W, G=G), W=W, G=G)


def test_many_batches():
    csrs = []
    for i in range(2500):
        n = 1 + (i * 7) % 13
        rp, c, v = tiny_batch(i, n_rows=n, n_cols=16, density=0.6, n_values=2,
                              prefix_copy=0.5)
        csrs.append((n, rp, c, v))
    B = _batches_from_csrs(csrs, 16)
    rng = np.random.default_rng(2)
    for k in (1, 8):
        W = rng.standard_normal((16, k)).astype(np.float32)
        G = rng.standard_normal((int(B.n_rows.sum()), k)).astype(np.float32)
        res = run_gpu(B, W=W, G=G, decode=(k == 1))
        check_against_oracle(B, res, W=W, G=G, batches=range(0, 2500, 97))
        if k == 1:
            rp_g, c_g, v_g = res["csr"]
            assert np.array_equal(rp_g, B.rowptr)
            assert np.array_equal(c_g, B.col)
            assert np.array_equal(v_g.view(np.uint32), B.val.view(np.uint32))


def test_left_run_to_run_within_tolerance():
    B = config_batches("c5", 0, 4)
    G = config_G("c5", 0, 4)
    a = run_gpu(B, G=G, decode=False)["out"]
    b = run_gpu(B, G=G, decode=False)["out"]
    scale = np.abs(a).max()
    assert np.max(np.abs(a - b)) <= 1e-5 * scale + 1e-30


def test_device_errors():
    B = _tiny_set(1)
    encs = T.toc_encode_batches(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    buf = torch.empty(T.toc_upload_size(encs), dtype=torch.uint8, device=DEV)
    dev = T.toc_upload(encs, buf)
    small = torch.empty(10, dtype=torch.uint8, device=DEV)
    with pytest.raises(T.TocError) as ei:
        T.toc_upload(encs, small)
    assert ei.value.status == T.TOC_ESIZE
    lib = T.lib()
    W = torch.zeros((B.n_cols, 4), device=DEV)
    R = torch.zeros((int(B.n_rows.sum()), 4), device=DEV)
    s = torch.cuda.current_stream().cuda_stream
    assert lib.toc_right_mul(dev.handle, W.data_ptr(), 0, 4, R.data_ptr(), 4, None, 0, s) \
        == T.TOC_EINVAL
    assert lib.toc_right_mul(dev.handle, W.data_ptr(), 4, 3, R.data_ptr(), 4, None, 0, s) \
        == T.TOC_EINVAL
    with pytest.raises(T.TocError):
        T.toc_right_mul(dev, W[:-1], R)
    B4 = config_batches("c4", 0, 1)
    encs = T.toc_encode_batches(B4.n_rows, B4.n_cols, B4.rowptr, B4.col, B4.val)
    buf = torch.empty(T.toc_upload_size(encs), dtype=torch.uint8, device=DEV)
    dev = T.toc_upload(encs, buf)
    W = torch.zeros((B4.n_cols, 8), device=DEV)
    R = torch.zeros((250, 8), device=DEV)
    ws_n, ws_min = T.toc_workspace_size(dev, T.TOC_OP_RIGHT, 8)
    assert ws_min > 0
    tiny_ws = torch.empty(ws_min // 8, dtype=torch.float32, device=DEV)
    with pytest.raises(T.TocError) as ei:
        T.toc_right_mul(dev, W, R, tiny_ws)
    assert ei.value.status == T.TOC_ESIZE
