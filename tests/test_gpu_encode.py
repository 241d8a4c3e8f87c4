"""GPU parity of the device encoder (Algorithm 1, section 3.1, after the sparse
encoding of section 3) with the oracle's encode: I, D and the node count of every
batch bit for bit, on tiny batches with repeats and explicit zeros, the worked
example, batches of every workload, and edge cases; malformed batches get their
status without disturbing the other batches of a launch."""

import json
import os

import numpy as np
import pytest

import oracle as O
import paper_1702_06943_amd as T
from workloads import Batches, config_batches, tiny_batch

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"
HERE = os.path.dirname(os.path.abspath(__file__))
GOLD = json.load(open(os.path.join(HERE, "golden", "worked_example.json")))


def encode_gpu(n_rows, n_cols, rowptr, col, val, max_nnz=None, ws=None):
    """Runs toc_encode_device over the concatenated CSR; returns, per batch, the
    tuple (I as (col, bits) pairs, D as lists of codes, node count, nonzeros) or
    None for a batch with a nonzero status, and the status array."""
    n_rows = np.asarray(n_rows, np.int32)
    rowptr = np.asarray(rowptr, np.int64)
    nb, nnz = n_rows.size, col.size
    if max_nnz is None:
        row_off = np.concatenate([[0], np.cumsum(n_rows)])
        max_nnz = int(max([rowptr[row_off[b + 1]] - rowptr[row_off[b]] for b in range(nb)]
                          + [0]))
    d_rp = torch.from_numpy(rowptr).to(DEV)
    d_col = torch.from_numpy(np.asarray(col, np.int32)).to(DEV)
    d_val = torch.from_numpy(np.asarray(val, np.float32)).to(DEV)
    I_col = torch.full((max(nnz, 1),), -7, dtype=torch.int32, device=DEV)
    I_val = torch.full((max(nnz, 1),), -7.0, dtype=torch.float32, device=DEV)
    D = torch.full((max(nnz, 1),), -7, dtype=torch.int32, device=DEV)
    D_rp = torch.full((int(n_rows.sum()) + nb,), -7, dtype=torch.int64, device=DEV)
    counts = torch.full((4 * nb,), -7, dtype=torch.int64, device=DEV)
    status = torch.full((nb,), -1, dtype=torch.int32, device=DEV)
    if ws is None:
        ws = torch.empty(max(T.toc_encode_device_workspace_size(nb, max_nnz), 1),
                         dtype=torch.uint8, device=DEV)
    T.toc_encode_device(n_rows, n_cols, d_rp, d_col, d_val, max_nnz, I_col, I_val, D, D_rp,
                        counts, status, ws)
    torch.cuda.synchronize()
    I_col, I_bits = I_col.cpu().numpy(), I_val.cpu().numpy().view(np.uint32)
    D, D_rp = D.cpu().numpy().view(np.uint32), D_rp.cpu().numpy()
    counts, status = counts.cpu().numpy().reshape(nb, 4), status.cpu().numpy()
    out, r = [], 0
    for b in range(nb):
        n = int(n_rows[b])
        if status[b] != 0:
            out.append(None)
            r += n
            continue
        s = int(rowptr[r] - rowptr[0])
        n_first, n_codes, n_nodes, nonzero = (int(x) for x in counts[b])
        I = [(int(c), int(v)) for c, v in zip(I_col[s:s + n_first], I_bits[s:s + n_first])]
        offs = D_rp[r + b:r + b + n + 1]
        assert offs[0] == 0 and offs[-1] == n_codes
        codes = D[s:s + n_codes]
        Dl = [[int(x) for x in codes[offs[i]:offs[i + 1]]] for i in range(n)]
        out.append((I, Dl, n_nodes, nonzero))
        r += n
    return out, status


def oracle_of(n, n_cols, rp, c, v):
    rows = O.canonicalize(n, n_cols, rp, c, v)
    I, D, N = O.encode(rows)
    return I, D, N, sum(len(t) for t in rows)


def assert_batches(B, got):
    for b in range(B.n_batches):
        n, rp, c, v = B.batch(b)
        assert got[b] is not None, f"batch {b} rejected"
        I, D, N, nz = oracle_of(n, B.n_cols, rp, c, v)
        gI, gD, gN, gnz = got[b]
        assert gI == I, f"batch {b}: I"
        assert gD == D, f"batch {b}: D"
        assert (gN, gnz) == (N, nz), f"batch {b}: counts"


def test_worked_example():
    rows_in = GOLD["rows_from_table2"]["rows"]
    rp = np.cumsum([0] + [len(r) for r in rows_in]).astype(np.int64)
    c = np.array([p[0] for r in rows_in for p in r], np.int32)
    v = np.array([p[1] for r in rows_in for p in r], np.float32)
    got, st = encode_gpu([len(rows_in)], GOLD["n_cols"], rp, c, v)
    assert st.tolist() == [0]
    I, D, N, _ = got[0]
    assert I == [(p[0], O.f32_bits(p[1])) for p in GOLD["I"]["pairs"]]
    assert D == GOLD["D"]["codes"]
    assert N == GOLD["sizes"]["n_nodes"]


def test_tiny_batches_in_one_launch():
    specs = [dict(n_rows=1, density=1.0, n_values=1), dict(n_rows=9, density=0.8, n_values=2,
             prefix_copy=0.6), dict(n_rows=25, density=0.9, n_values=2, prefix_copy=0.9),
             dict(n_rows=40, density=0.3, n_values=5), dict(n_rows=16, density=1.0, n_values=1),
             dict(n_rows=3, density=0.0, n_values=1)]
    parts = []
    for seed in range(12):
        for k, spec in enumerate(specs):
            rp, c, v = tiny_batch(7000 + 31 * seed + k, n_cols=12, zeros=(seed % 2 == 0),
                                  **spec)
            parts.append(Batches(12, [spec["n_rows"]], rp, c, v))
    B = Batches.concat(parts)
    got, st = encode_gpu(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    assert (st == 0).all()
    assert_batches(B, got)


@pytest.mark.parametrize("cfg,first,nb", [("c1", 0, 1), ("c2", 5, 3), ("c3", 11, 2),
                                          ("c4", 2, 1), ("c5", 40, 16)])
def test_workload_batches_vs_oracle(cfg, first, nb):
    B = config_batches(cfg, first, nb)
    got, st = encode_gpu(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    assert (st == 0).all()
    assert_batches(B, got)


@pytest.mark.parametrize("cfg,nb", [("c3", 96), ("c5", 300), ("c2", 40)])
def test_many_batches_vs_host_encoder(cfg, nb):
    """The host encoder is pinned to the oracle by the CPU tests; here it checks
    launches of many batches."""
    B = config_batches(cfg, 0, nb)
    got, st = encode_gpu(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    assert (st == 0).all()
    encs = T.toc_encode_batches(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    for b in range(nb):
        I_col, I_val, D_rp, D_codes = T.toc_enc_export(encs[b])
        gI, gD, gN, _ = got[b]
        assert gI == [(int(c), int(v)) for c, v in zip(I_col, I_val.view(np.uint32))]
        assert [x for d in gD for x in d] == D_codes.tolist()
        assert np.array_equal(np.cumsum([0] + [len(d) for d in gD]), D_rp)
        assert gN == T.toc_enc_info_get(encs[b])["n_nodes"]


def test_lanes_and_groups_take_several_batches():
    """A large declared max_nnz leaves room for 64 tables per phase, so each
    workgroup and each lane encodes several of the 150 batches in turn."""
    parts = []
    for k in range(150):
        rp, c, v = tiny_batch(9100 + k, n_rows=1 + k % 23, n_cols=10, density=0.7,
                              n_values=2, zeros=(k % 5 == 0), prefix_copy=0.5)
        parts.append(Batches(10, [1 + k % 23], rp, c, v))
    B = Batches.concat(parts)
    got, st = encode_gpu(B.n_rows, B.n_cols, B.rowptr, B.col, B.val, max_nnz=1 << 22)
    assert (st == 0).all()
    assert_batches(B, got)


def test_edge_cases():
    """A batch without rows, an all-zero batch, empty rows, one-entry rows, and a
    row pointer that does not start at 0."""
    n_rows = [0, 3, 4, 1, 0]
    rowptr = np.array([0, 2, 2, 3,   3, 3, 4, 4,   5], np.int64)
    col = np.array([0, 3, 1,   2,   4], np.int32)
    val = np.array([0.0, -0.0, 0.0,   1.5,   1.5], np.float32)
    B = Batches(5, n_rows, rowptr, col, val)
    for shift in (0, 1000):
        got, st = encode_gpu(n_rows, 5, rowptr + shift, col, val)
        assert st.tolist() == [0] * 5
        assert got[0] == ([], [], 1, 0)
        assert got[1] == ([], [[], [], []], 1, 0)
        assert got[2] == ([(2, O.f32_bits(1.5))], [[], [], [1], []], 2, 1)
        assert got[3] == ([(4, O.f32_bits(1.5))], [[1]], 2, 1)
        assert got[4] == ([], [], 1, 0)
        assert_batches(B, got)


def test_malformed_batches_get_status():
    good = config_batches("c5", 0, 3)
    parts = [good]
    for bad in ("col", "nan", "range"):
        rp, c, v = tiny_batch(4242, n_rows=6, n_cols=12, density=0.8, n_values=2)
        c, v = c.copy(), v.copy()
        if bad == "col":                        # a repeated column inside a row
            i = next(i for i in range(6) if rp[i + 1] - rp[i] >= 2)
            c[rp[i] + 1] = c[rp[i]]
        elif bad == "nan":
            v[5] = np.nan
        else:
            c[-1] = good.n_cols
        parts.append(Batches(good.n_cols, [6], rp, c, v))
    parts.append(config_batches("c5", 3, 2))
    B = Batches.concat(parts)
    got, st = encode_gpu(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    assert st.tolist() == [0, 0, 0, T.TOC_ENCDEV_COLUMN, T.TOC_ENCDEV_VALUE,
                           T.TOC_ENCDEV_COLUMN, 0, 0]
    ok = [got[b] for b in (0, 1, 2, 6, 7)]
    assert_batches(Batches.concat([good, config_batches("c5", 3, 2)]), ok)
    # batches above the declared max_nnz
    B = config_batches("c2", 0, 3)
    sizes = [int(B.batch(b)[1][-1]) for b in range(3)]
    mid = sorted(sizes)[1]
    got, st = encode_gpu(B.n_rows, B.n_cols, B.rowptr, B.col, B.val, max_nnz=mid)
    for b in range(3):
        assert st[b] == (T.TOC_ENCDEV_SIZE if sizes[b] > mid else 0)
        if sizes[b] <= mid:
            n, rp, c, v = B.batch(b)
            assert got[b][:3] == oracle_of(n, B.n_cols, rp, c, v)[:3]


def test_decreasing_rowptr_between_batches():
    """A tuple of negative length at the end of batch 0: batch 0 fails its own
    row check, batch 1 the check of its start against batch 0's last row."""
    B = config_batches("c5", 0, 3)
    rp = B.rowptr.copy()
    r = int(B.n_rows[0])
    rp[r] = rp[r - 1] - 1
    got, st = encode_gpu(B.n_rows, B.n_cols, rp, B.col, B.val)
    assert st.tolist() == [T.TOC_ENCDEV_ROWPTR, T.TOC_ENCDEV_ROWPTR, 0]
    n, brp, c, v = B.batch(2)
    assert got[2][:3] == oracle_of(n, B.n_cols, brp, c, v)[:3]


def test_workspace_reused_by_a_second_call():
    """The child tables keep the first call's entries; the second call must not
    read them (the same batch indexes, other data, fewer entries)."""
    A = config_batches("c3", 0, 4)
    B = config_batches("c5", 7, 4)
    max_nnz = max(int(A.batch(b)[1][-1]) for b in range(4))
    ws = torch.empty(T.toc_encode_device_workspace_size(4, max_nnz), dtype=torch.uint8,
                     device=DEV)
    got, st = encode_gpu(A.n_rows, A.n_cols, A.rowptr, A.col, A.val, max_nnz=max_nnz, ws=ws)
    assert (st == 0).all()
    assert_batches(A, got)
    got, st = encode_gpu(B.n_rows, B.n_cols, B.rowptr, B.col, B.val, max_nnz=max_nnz, ws=ws)
    assert (st == 0).all()
    assert_batches(B, got)
