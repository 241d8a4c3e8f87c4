"""Pins of the CPU oracle against facts the paper and the mathematics fix.

Nothing here compares the oracle with itself: every check is against the paper's
worked example (tests/golden/worked_example.json), a brute-force re-encoder written
from the definition of greedy longest-prefix matching, numpy's dense matmul on the
densified batch, integer exactness, closed-form counts, or the lossless round trip.
"""

import json
import os

import numpy as np
import pytest

import oracle as O
from workloads import tiny_batch

HERE = os.path.dirname(os.path.abspath(__file__))
GOLD = json.load(open(os.path.join(HERE, "golden", "worked_example.json")))


def _pairs(lst):
    return [(int(c), O.f32_bits(v)) for c, v in lst]


def _rows_to_csr(rows):
    rowptr = [0]
    col, val = [], []
    for r in rows:
        for c, v in r:
            col.append(c)
            val.append(v)
        rowptr.append(len(col))
    return np.array(rowptr), np.array(col, np.int32), np.array(val, np.float32)


def _dense(rows, n_cols):
    A = np.zeros((len(rows), n_cols))
    for i, r in enumerate(rows):
        for c, b in r:
            A[i, c] = O.bits_f32(b)
    return A


@pytest.fixture(scope="module")
def example():
    rows_in = GOLD["rows_from_table2"]["rows"]
    rp, c, v = _rows_to_csr(rows_in)
    rows = O.canonicalize(len(rows_in), GOLD["n_cols"], rp, c, v)
    I, D, N = O.encode(rows)
    return rows, I, D, N


# --- worked example (Table 2, Table 4, Section 3) ---------------------------------
def test_sparse_encoding_example_row():
    # Section 3: dense tuple [1.1, 2, 3, 0] -> [1:1.1, 2:2, 3:3] (0-based here)
    rows = O.canonicalize(1, 4, [0, 4], [0, 1, 2, 3],
                          np.array([1.1, 2, 3, 0], np.float32))
    assert rows == [_pairs([[0, 1.1], [1, 2.0], [2, 3.0]])]


def test_worked_example_I_and_D(example):
    rows, I, D, N = example
    assert I == _pairs(GOLD["I"]["pairs"])
    assert D == GOLD["D"]["codes"]
    assert N == GOLD["sizes"]["n_nodes"]


def test_worked_example_cprime(example):
    rows, I, D, N = example
    cp = O.build_cprime(I, D)
    want_key = GOLD["cprime"]["key"]
    want_par = GOLD["cprime"]["parent"]
    assert cp["n_nodes"] == len(want_key)
    for i in range(1, cp["n_nodes"]):
        assert cp["key"][i] == (want_key[i][0], O.f32_bits(want_key[i][1])), i
        assert cp["parent"][i] == want_par[i], i


def test_worked_example_added_sequences(example):
    rows, I, D, N = example
    cp = O.build_cprime(I, D)
    for node, seq in GOLD["added_nodes"]["sequences"].items():
        node = int(node)
        got = []
        while node != 0:
            got.append(cp["key"][node])
            node = cp["parent"][node]
        assert got[::-1] == _pairs(seq)


def test_worked_example_decode(example):
    rows, I, D, N = example
    assert O.decode(I, D) == rows
    assert rows == [_pairs(r) for r in GOLD["rows_from_table2"]["rows"]]


def test_worked_example_products(example):
    rows, I, D, N = example
    ones_w = np.ones((4, 1), np.float32)
    ones_g = np.ones((4, 1), np.float32)
    R, _ = O.dense_right(rows, 4, ones_w)
    out, _ = O.dense_left(rows, 4, ones_g)
    # values 1.1 and 1.4 are binary32-rounded, so compare loosely with the hand sums
    assert np.allclose(R[:, 0], GOLD["products_all_ones"]["right"], rtol=0, atol=1e-6)
    assert np.allclose(out[:, 0], GOLD["products_all_ones"]["left"], rtol=0, atol=1e-6)
    assert np.allclose(O.toc_right(I, D, ones_w), R, rtol=0, atol=1e-12)
    assert np.allclose(O.toc_left(I, D, ones_g, 4), out, rtol=0, atol=1e-12)


def test_worked_example_sizes(example):
    rows, I, D, N = example
    st = O.layout_stats(I, D)
    s = GOLD["sizes"]
    assert st["n_live"] == s["n_live"]
    assert st["n_deep"] == s["n_deep"]
    assert st["max_depth"] == s["max_depth"]
    assert st["n_nodes"] == s["n_nodes"]
    assert st["canon_bytes"] == s["canon_bytes"]
    assert O.physical_bytes(I, D) == s["physical_bytes"]


def test_worked_example_variant_sizes(example):
    rows, I, D, N = example
    v = GOLD["variant_sizes"]
    assert O.dense_bytes(4, 4) == v["dense_bytes"]
    assert O.sparse_bytes(rows) == v["sparse_bytes"]
    assert O.logical_bytes(I, D) == v["logical_bytes"]


# --- brute-force re-encoder -------------------------------------------------------
def brute_force_encode(rows):
    """Greedy longest-prefix dictionary coding written from its definition, with a
    dict of whole sequences instead of a tree: at each position try every length
    from the longest down and take the first one present in the dictionary."""
    seqs = {}
    I = []
    for t in rows:
        for p in t:
            if (p,) not in seqs:
                seqs[(p,)] = len(seqs) + 1
                I.append(p)
    D = []
    for t in rows:
        i, codes = 0, []
        while i < len(t):
            for L in range(len(t) - i, 0, -1):
                s = tuple(t[i:i + L])
                if s in seqs:
                    break
            codes.append(seqs[s])
            if i + L < len(t):
                seqs[s + (t[i + L],)] = len(seqs) + 1
            i += L
        D.append(codes)
    return I, D, len(seqs) + 1


CASES = [
    dict(n_rows=1, n_cols=1, density=1.0, n_values=1),
    dict(n_rows=6, n_cols=5, density=0.7, n_values=2),
    dict(n_rows=8, n_cols=8, density=0.9, n_values=2, prefix_copy=0.5),
    dict(n_rows=12, n_cols=6, density=1.0, n_values=1),
    dict(n_rows=20, n_cols=10, density=0.5, n_values=3, prefix_copy=0.7),
    dict(n_rows=7, n_cols=30, density=0.2, n_values=4),
    dict(n_rows=30, n_cols=12, density=0.8, n_values=2, prefix_copy=0.9),
]


@pytest.mark.parametrize("seed", range(12))
@pytest.mark.parametrize("case", range(len(CASES)))
def test_encoder_matches_brute_force(seed, case):
    rp, c, v = tiny_batch(seed * 31 + case, **CASES[case])
    spec = CASES[case]
    rows = O.canonicalize(spec["n_rows"], spec["n_cols"], rp, c, v)
    I, D, N = O.encode(rows)
    I2, D2, N2 = brute_force_encode(rows)
    assert (I, D, N) == (I2, D2, N2)


# --- round trip and C' invariants ----------------------------------------------
@pytest.mark.parametrize("seed", range(10))
@pytest.mark.parametrize("case", range(len(CASES)))
def test_round_trip_and_invariants(seed, case):
    spec = CASES[case]
    rp, c, v = tiny_batch(1000 + seed * 31 + case, zeros=True, **spec)
    rows = O.canonicalize(spec["n_rows"], spec["n_cols"], rp, c, v)
    # zeros dropped, everything else kept
    keep = np.asarray(v) != 0
    assert sum(len(r) for r in rows) == int(keep.sum())
    I, D, N = O.encode(rows)
    assert O.decode(I, D) == rows
    cp = O.build_cprime(I, D)
    # node count: |I| roots-children plus one node per non-final code of each row
    assert cp["n_nodes"] == N == 1 + len(I) + sum(max(len(d) - 1, 0) for d in D)
    seen = {}
    for i in range(1, N):
        p = cp["parent"][i]
        assert 0 <= p < i
        assert cp["depth"][i] == (cp["depth"][p] + 1 if p else 1)
        k = (p, cp["key"][i])
        assert k not in seen, "siblings must have distinct keys"
        seen[k] = i
    # each row: code depths add up to the row length; each code covers a run of
    # strictly increasing columns
    for r, d in zip(rows, D):
        assert sum(cp["depth"][x] for x in d) == len(r)


def test_encode_empty_and_all_zero():
    rows = O.canonicalize(0, 5, [0], [], np.zeros(0, np.float32))
    assert O.encode(rows) == ([], [], 1)
    rows = O.canonicalize(3, 4, [0, 2, 2, 3], [0, 3, 1],
                          np.array([0.0, -0.0, 0.0], np.float32))
    I, D, N = O.encode(rows)
    assert (I, D, N) == ([], [[], [], []], 1)
    st = O.layout_stats(I, D)
    assert st["n_live"] == 0 and st["max_depth"] == 0
    assert st["canon_bytes"] == 4 * 0 + 4 * 4 + 0 + 4


@pytest.mark.parametrize("bad", [
    dict(rowptr=[0, 2], col=[1, 1], val=[1, 2]),          # duplicate column
    dict(rowptr=[0, 2], col=[2, 1], val=[1, 2]),          # unsorted
    dict(rowptr=[0, 1], col=[4], val=[1]),                # out of range
    dict(rowptr=[0, 1], col=[0], val=[np.nan]),
    dict(rowptr=[0, 1], col=[0], val=[np.inf]),
    dict(rowptr=[1, 1], col=[], val=[]),                  # rowptr[0] != 0
    dict(rowptr=[0, 2], col=[0], val=[1]),                # length mismatch
])
def test_canonicalize_rejects(bad):
    with pytest.raises(O.TocInputError):
        O.canonicalize(1, 4, bad["rowptr"], bad["col"], np.array(bad["val"], np.float32))


# --- products: Theorems 1 and 2, numpy matmul, integers, duality ---------------
@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("case", range(len(CASES)))
@pytest.mark.parametrize("k", [1, 3])
def test_products(seed, case, k):
    spec = CASES[case]
    integer = seed % 2 == 0
    rp, c, v = tiny_batch(2000 + seed * 31 + case, integer=integer, **spec)
    rows = O.canonicalize(spec["n_rows"], spec["n_cols"], rp, c, v)
    I, D, N = O.encode(rows)
    rng = np.random.default_rng(seed)
    if integer:
        W = rng.integers(-4, 5, size=(spec["n_cols"], k)).astype(np.float32)
        G = rng.integers(-4, 5, size=(spec["n_rows"], k)).astype(np.float32)
    else:
        W = rng.standard_normal((spec["n_cols"], k)).astype(np.float32)
        G = rng.standard_normal((spec["n_rows"], k)).astype(np.float32)
    A = _dense(rows, spec["n_cols"])
    assert np.array_equal(O.densify(rows, spec["n_cols"]), A)
    R, SR = O.dense_right(rows, spec["n_cols"], W)
    out, SO = O.dense_left(rows, spec["n_cols"], G)
    R_np = A @ W.astype(np.float64)
    out_np = A.T @ G.astype(np.float64)
    R_toc = O.toc_right(I, D, W)
    out_toc = O.toc_left(I, D, G, spec["n_cols"])
    if integer:
        assert np.array_equal(R, R_np) and np.array_equal(R_toc, R_np)
        assert np.array_equal(out, out_np) and np.array_equal(out_toc, out_np)
    else:
        tol_r = 1e-12 * SR + 1e-300
        tol_o = 1e-12 * SO + 1e-300
        assert np.all(np.abs(R - R_np) <= tol_r)
        assert np.all(np.abs(R_toc - R_np) <= tol_r)
        assert np.all(np.abs(out - out_np) <= tol_o)
        assert np.all(np.abs(out_toc - out_np) <= tol_o)
    assert np.all(SR >= np.abs(R) - 1e-12) and np.all(SO >= np.abs(out) - 1e-12)
    # duality <G, A W> = <A^T G, W>
    lhs = float(np.sum(G.astype(np.float64) * R))
    rhs = float(np.sum(out * W.astype(np.float64)))
    assert abs(lhs - rhs) <= 1e-9 * (1 + abs(lhs))


def test_scale_is_zero_only_for_structural_zeros():
    rows = O.canonicalize(2, 3, [0, 1, 1], [1], np.array([2.0], np.float32))
    W = np.ones((3, 2), np.float32)
    R, S = O.dense_right(rows, 3, W)
    assert np.all(S[1] == 0) and np.all(R[1] == 0) and np.all(S[0] == 2)


# --- sparse-safe element-wise ops (Algorithm 3) and A .+ c (Algorithm 9) ----------
def _csr_arrays(rows):
    """rows of (col, bits) -> (row index, col, float32 value) arrays."""
    ri = np.asarray([i for i, r in enumerate(rows) for _ in r], dtype=np.int64)
    ci = np.asarray([c for r in rows for c, _ in r], dtype=np.int64)
    vi = np.asarray([b for r in rows for _, b in r], dtype=np.uint32).view(np.float32)
    return ri, ci, vi


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("case", range(len(CASES)))
@pytest.mark.parametrize("op,c", [(0, 1.0), (0, -1.0), (0, 2.0), (0, 0.37), (0, 0.0), (1, 0.0)])
def test_map_values_commutes_with_decode(seed, case, op, c):
    # Algorithm 3 changes only I; the section's claim is that this applies the
    # element-wise op to every nonzero of A.  Checked against the op applied by
    # numpy to the decoded values (vectorised binary32 arithmetic).
    spec = CASES[case]
    rp, col, val = tiny_batch(2000 + seed * 31 + case, **spec)
    rows = O.canonicalize(spec["n_rows"], spec["n_cols"], rp, col, val)
    I, D, _ = O.encode(rows)
    got = _csr_arrays(O.decode(O.map_values(I, op, c), D))
    ri, ci, vi = _csr_arrays(rows)
    want = vi * np.float32(c) if op == O.MAP_SCALE else vi * vi
    assert np.array_equal(got[0], ri) and np.array_equal(got[1], ci)
    assert np.array_equal(got[2].view(np.uint32), want.astype(np.float32).view(np.uint32))


def test_map_values_exact_cases():
    rows = [[(0, O.f32_bits(1.5)), (3, O.f32_bits(-2.25))], [(1, O.f32_bits(3.0))]]
    I, D, _ = O.encode(rows)
    bits = np.asarray([b for _, b in I], dtype=np.uint32)
    # c = 1: identical bits; c = -1: only the sign bit flips; c = 2: exponent + 1
    assert [b for _, b in O.map_values(I, O.MAP_SCALE, 1.0)] == bits.tolist()
    assert [b for _, b in O.map_values(I, O.MAP_SCALE, -1.0)] == (bits ^ 0x80000000).tolist()
    assert [b for _, b in O.map_values(I, O.MAP_SCALE, 2.0)] == (bits + (1 << 23)).tolist()
    # squares of small integers are exact
    rows = [[(0, O.f32_bits(3.0)), (1, O.f32_bits(-7.0))], [(0, O.f32_bits(12.0))]]
    I, D, _ = O.encode(rows)
    sq = [O.bits_f32(b) for _, b in O.map_values(I, O.MAP_SQUARE)]
    assert sq == [O.bits_f32(b) ** 2 for _, b in I]
    assert [c for c, _ in O.map_values(I, O.MAP_SQUARE)] == [c for c, _ in I]


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("case", range(len(CASES)))
def test_dense_plus(seed, case):
    spec = CASES[case]
    rp, col, val = tiny_batch(3000 + seed * 31 + case, zeros=True, **spec)
    n, m = spec["n_rows"], spec["n_cols"]
    rows = O.canonicalize(n, m, rp, col, val)
    ri, ci, vi = _csr_arrays(rows)
    # c = 0: the dense matrix has exactly the CSR's nonzeros
    A = O.dense_plus(rows, m, 0.0)
    assert A.dtype == np.float32 and A.shape == (n, m)
    nz = np.nonzero(A)
    assert np.array_equal(nz[0], ri) and np.array_equal(nz[1], ci)
    assert np.array_equal(A[nz].view(np.uint32), vi.view(np.uint32))
    # c != 0: zeros become c, every stored entry a + c
    c = np.float32(-1.25)
    B = O.dense_plus(rows, m, c)
    mask = np.ones((n, m), bool)
    mask[ri, ci] = False
    assert np.all(B[mask] == c)
    assert np.array_equal(B[ri, ci], (vi + c).astype(np.float32))


def test_dense_plus_integer_sum():
    # integer-valued A and c: every element is exact, so the total is closed-form
    rng = np.random.default_rng(5)
    n, m = 9, 13
    dense = rng.integers(-4, 5, size=(n, m)).astype(np.float32)
    dense[rng.random((n, m)) < 0.4] = 0
    rp = np.concatenate([[0], np.cumsum((dense != 0).sum(1))]).astype(np.int64)
    col = np.concatenate([np.flatnonzero(r) for r in dense]).astype(np.int32)
    val = dense[dense != 0].astype(np.float32)
    rows = O.canonicalize(n, m, rp, col, val)
    I, D, _ = O.encode(rows)
    B = O.dense_plus(O.decode(I, D), m, 3.0)
    assert float(B.astype(np.float64).sum()) == float(dense.sum()) + 3.0 * n * m


# --- physical encoding (Section 3.2) as bytes --------------------------------------
PHYS = json.load(open(os.path.join(HERE, "golden", "physical_worked_example.json")))


def test_physical_worked_example(example):
    rows, I, D, N = example
    want = bytes.fromhex("".join(a["hex"] for a in PHYS["arrays"]))
    assert len(want) == PHYS["total_bytes"] == GOLD["sizes"]["physical_bytes"]
    assert O.pack_physical(I, D) == want
    assert O.unpack_physical(want) == (I, D)


# Section 3.2's width rule at each byte boundary; its own example: a largest column
# index of 4 needs 1 byte
@pytest.mark.parametrize("mx,width,tail", [
    (0, 1, "00"), (4, 1, "04"), (255, 1, "ff"), (256, 2, "0001"), (65535, 2, "ffff"),
    (65536, 3, "000001"), (0x123456, 3, "563412"), (2**24 - 1, 3, "ffffff"),
    (2**24, 4, "00000001"), (2**32 - 1, 4, "ffffffff")])
def test_physical_width_rule(mx, width, tail):
    blob = O.pack_physical([(mx, O.f32_bits(1.0))], [])
    # the I-column array: count 1, then the width, then the column in that many bytes
    assert blob[:5 + width].hex() == "01000000" + "%02x" % width + tail
    assert O.unpack_physical(blob) == ([(mx, O.f32_bits(1.0))], [])


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("case", range(len(CASES)))
def test_physical_round_trip(seed, case):
    spec = CASES[case]
    rp, c, v = tiny_batch(3000 + seed * 31 + case, **spec)
    rows = O.canonicalize(spec["n_rows"], spec["n_cols"], rp, c, v)
    I, D, N = O.encode(rows)
    blob = O.pack_physical(I, D)
    assert len(blob) == O.physical_bytes(I, D)
    assert O.unpack_physical(blob) == (I, D)
    assert O.decode(*O.unpack_physical(blob)) == rows


def test_physical_empty_batch():
    blob = O.pack_physical([], [[], []])
    assert O.unpack_physical(blob) == ([], [[], []])
    assert O.build_cprime(*O.unpack_physical(blob))["n_nodes"] == 1


def _phys_example():
    return bytearray(bytes.fromhex("".join(a["hex"] for a in PHYS["arrays"])))


def _bad_truncated():
    return _phys_example()[:-1]


def _bad_trailing():
    return _phys_example() + b"\x00"


def _bad_width():
    b = _phys_example()
    b[4] = 5
    return b


def _bad_value_width():
    b = _phys_example()
    b[10 + 4] = 2
    return b


def _bad_value_index():
    b = _phys_example()
    b[10 + 21 + 5] = 4          # first value index -> 4, but only 4 unique values
    return b


def _bad_starts():
    b = _phys_example()
    b[-3] = 7                   # tuple starts 0,4,7,6,9: not monotone
    b[-2] = 6
    return b


@pytest.mark.parametrize("make", [_bad_truncated, _bad_trailing, _bad_width,
                                  _bad_value_width, _bad_value_index, _bad_starts])
def test_physical_rejects(make):
    with pytest.raises(O.TocInputError):
        O.unpack_physical(bytes(make()))


# --- mini-batch gradient descent step (section 2.1) --------------------------------
def _mean_loss(A, h, y, loss):
    return float(np.mean(O.mgd_loss(loss, A @ h, y)))


@pytest.mark.parametrize("loss", [O.MGD_LINEAR, O.MGD_LOGISTIC, O.MGD_HINGE])
@pytest.mark.parametrize("seed", range(4))
def test_mgd_step_is_gradient_step(loss, seed):
    """h - h_new = lr * grad of the mean loss, the gradient taken by central finite
    differences of the loss definitions on the densified batch."""
    spec = dict(n_rows=12, n_cols=7, density=0.6, n_values=3)
    rp, c, v = tiny_batch(4000 + seed, **spec)
    rows = O.canonicalize(12, 7, rp, c, v)
    A = _dense(rows, 7)
    rng = np.random.default_rng(seed)
    for _ in range(100):                     # keep every margin away from the hinge's kink
        h = rng.standard_normal(7) * 0.3
        y = rng.choice([-1.0, 1.0], size=12)
        if np.all(np.abs(y * (A @ h) - 1.0) > 1e-3):
            break
    lr = 0.37
    h_new, _ = O.mgd_step(rows, 7, h, y, loss, lr)
    eps = 1e-6
    fd = np.array([(_mean_loss(A, h + eps * e, y, loss) - _mean_loss(A, h - eps * e, y, loss))
                   / (2 * eps) for e in np.eye(7)])
    assert np.allclose((h - h_new) / lr, fd, rtol=1e-6, atol=1e-8)


def test_mgd_linear_worked_example(example):
    """Section 2.1's linear-regression gradient ((A h - Y)^T A)^T on the example
    table, summed by hand: h = 1, Y = (1, 2, 3, 4) give A h - Y = (6.5, 4.1, 2.5,
    -0.9) and the gradient (10.67, 22.15, 39.3, 12.6); lr = 0.1 over 4 tuples."""
    rows = example[0]
    h_new, _ = O.mgd_step(rows, 4, np.ones(4), np.array([1.0, 2, 3, 4]), O.MGD_LINEAR, 0.1)
    assert np.allclose(h_new, 1 - 0.025 * np.array([10.67, 22.15, 39.3, 12.6]), atol=2e-6)


def test_mgd_closed_forms():
    one = [[(2, O.f32_bits(1.5))]]
    h = np.array([0.0, 0.0, 0.25])
    # linear, one entry: h_j - lr (a h_j - y) a
    h1, _ = O.mgd_step(one, 3, h, np.array([2.0]), O.MGD_LINEAR, 0.5)
    assert h1.tolist() == [0.0, 0.0, 0.25 - 0.5 * (1.5 * 0.25 - 2.0) * 1.5]
    # logistic at r = 0: g = -y / 2
    h2, _ = O.mgd_step(one, 3, np.zeros(3), np.array([1.0]), O.MGD_LOGISTIC, 1.0)
    assert h2.tolist() == [0.0, 0.0, 0.75]
    # hinge beyond the margin: no change; inside: h + lr y a
    h3, _ = O.mgd_step(one, 3, np.array([0.0, 0.0, 1.0]), np.array([1.0]), O.MGD_HINGE, 1.0)
    assert h3.tolist() == [0.0, 0.0, 1.0]
    h4, _ = O.mgd_step(one, 3, np.zeros(3), np.array([-1.0]), O.MGD_HINGE, 2.0)
    assert h4.tolist() == [0.0, 0.0, -3.0]
    # lr = 0 and an empty batch change nothing
    assert O.mgd_step(one, 3, h, np.array([5.0]), O.MGD_LINEAR, 0.0)[0].tolist() == h.tolist()
    assert O.mgd_step([], 3, h, np.array([]), O.MGD_LINEAR, 1.0)[0].tolist() == h.tolist()


def test_mgd_tolerance_scale_is_absolute():
    """The scale is |A|^T (|g| + |A||h|): nonnegative, and on one entry a at column j
    equal to |a| (|g| + |a h_j|)."""
    rows = [[(0, O.f32_bits(-2.0))], [(0, O.f32_bits(3.0)), (1, O.f32_bits(-1.0))]]
    h = np.array([0.5, -4.0])
    y = np.array([1.0, -2.0])
    _, scale = O.mgd_step(rows, 2, h, y, O.MGD_LINEAR, 1.0)
    g = np.array([-2.0 * 0.5 - 1.0, 3.0 * 0.5 + 4.0 + 2.0])
    s_r = np.array([1.0, 1.5 + 4.0])
    assert np.allclose(scale, [2.0 * (abs(g[0]) + s_r[0]) + 3.0 * (abs(g[1]) + s_r[1]),
                               1.0 * (abs(g[1]) + s_r[1])])


# --- neural network step (section 5.1's network, Table 1's A.M and M.A) -------------
def _mlp_params(rng, m, h1, h2, C, scale=0.5):
    return {"W1": rng.standard_normal((m, h1)) * scale, "b1": rng.standard_normal(h1) * scale,
            "W2": rng.standard_normal((h1, h2)) * scale, "b2": rng.standard_normal(h2) * scale,
            "W3": rng.standard_normal((h2, C)) * scale, "b3": rng.standard_normal(C) * scale}


@pytest.mark.parametrize("C", [1, 3])
@pytest.mark.parametrize("seed", range(3))
def test_mlp_step_is_gradient_step(C, seed):
    """p - p_new = lr * d(mean loss)/dp for every entry of every parameter, the
    derivative taken by central finite differences of the loss definition."""
    rp, c, v = tiny_batch(4300 + seed, n_rows=9, n_cols=7, density=0.6, n_values=3)
    rows = O.canonicalize(9, 7, rp, c, v)
    rng = np.random.default_rng(seed)
    p = _mlp_params(rng, 7, 4, 3, C)
    labels = rng.integers(0, max(C, 2), size=9)
    lr = 0.3
    new, g = O.mlp_step(rows, 7, p, labels, lr)
    eps = 1e-6
    for name, val in p.items():
        for idx in np.ndindex(val.shape):
            hi = {k: x.copy() for k, x in p.items()}
            lo = {k: x.copy() for k, x in p.items()}
            hi[name][idx] += eps
            lo[name][idx] -= eps
            fd = (O.mlp_loss(rows, 7, hi, labels) - O.mlp_loss(rows, 7, lo, labels)) / (2 * eps)
            assert abs(g[name][idx] - fd) <= 1e-6 * abs(fd) + 1e-9, (name, idx)
            assert abs((val[idx] - new[name][idx]) / lr - fd) <= 1e-6 * abs(fd) + 1e-9


def test_mlp_closed_form_at_zero_weights():
    """All weights and biases 0: every hidden unit is 1/2 and the output uniform, so
    d/db3_c = (1/C - [y = c]) averaged over the tuples, d/dW3[u, c] = d/db3_c / 2, and
    every other gradient is 0 (W3 = 0 stops the backward pass)."""
    rows = [[(0, O.f32_bits(1.0)), (2, O.f32_bits(-2.0))], [(1, O.f32_bits(3.0))],
            [(2, O.f32_bits(0.5))], []]
    p = {"W1": np.zeros((3, 4)), "b1": np.zeros(4), "W2": np.zeros((4, 2)), "b2": np.zeros(2),
         "W3": np.zeros((2, 3)), "b3": np.zeros(3)}
    labels = np.array([0, 2, 2, 1])
    new, g = O.mlp_step(rows, 3, p, labels, 1.0)
    db3 = np.array([1 / 3 - 1 / 4, 1 / 3 - 1 / 4, 1 / 3 - 2 / 4])
    assert np.allclose(g["b3"], db3, rtol=0, atol=1e-15)
    assert np.allclose(g["W3"], np.tile(db3 / 2, (2, 1)), rtol=0, atol=1e-15)
    for k in ("W1", "b1", "W2", "b2"):
        assert not g[k].any()
    assert np.allclose(new["b3"], -db3, rtol=0, atol=1e-15)
    # one sigmoid output: at z = 0 the gradient of the bias is the mean of 1/2 - y
    p1 = dict(p, W3=np.zeros((2, 1)), b3=np.zeros(1))
    _, g1 = O.mlp_step(rows, 3, p1, np.array([1, 0, 1, 1]), 1.0)
    assert np.allclose(g1["b3"], [0.5 - 0.75], rtol=0, atol=1e-15)


@pytest.mark.parametrize("C", [1, 3])
@pytest.mark.parametrize("seed", range(3))
def test_mlp_grad_scale_bounds_the_gradient(C, seed):
    """S >= |g| for every entry of every gradient (the scale sums the absolute
    values of the terms the gradient sums)."""
    rp, c, v = tiny_batch(4400 + seed, n_rows=11, n_cols=6, density=0.6, n_values=3)
    rows = O.canonicalize(11, 6, rp, c, v)
    rng = np.random.default_rng(seed)
    p = _mlp_params(rng, 6, 5, 3, C)
    labels = rng.integers(0, max(C, 2), size=11)
    _, g = O.mlp_step(rows, 6, p, labels, 1.0)
    S = O.mlp_grad_scale(rows, 6, p, labels)
    for k in g:
        assert S[k].shape == g[k].shape
        assert np.all(S[k] >= np.abs(g[k]) * (1 - 1e-12)), k
        assert np.any(S[k] > np.abs(g[k]) * (1 + 1e-9)) or not g[k].any() or C == 1, k


def test_mlp_grad_scale_at_zero_weights():
    """Zero weights and biases: no forward rounding (c = 0), hidden units 1/2, the
    output uniform, and W3 = 0 stops the backward pass; so only the output layer
    has a scale, that of b3_c being the mean over the tuples of |1/C - [y = c]|
    and that of W3[u, c] half of it."""
    rows = [[(0, O.f32_bits(1.0)), (2, O.f32_bits(-2.0))], [(1, O.f32_bits(3.0))],
            [(2, O.f32_bits(0.5))], []]
    p = {"W1": np.zeros((3, 4)), "b1": np.zeros(4), "W2": np.zeros((4, 2)), "b2": np.zeros(2),
         "W3": np.zeros((2, 3)), "b3": np.zeros(3)}
    labels = np.array([0, 2, 2, 1])
    S = O.mlp_grad_scale(rows, 3, p, labels)
    # class 0: one tuple of it (|1/3 - 1|) and three others (1/3 each); class 1
    # likewise; class 2: two tuples of it and two others
    sb3 = np.array([(2 / 3 + 3 * 1 / 3) / 4, (2 / 3 + 3 * 1 / 3) / 4, (2 * 2 / 3 + 2 * 1 / 3) / 4])
    assert np.allclose(S["b3"], sb3, rtol=0, atol=1e-15)
    assert np.allclose(S["W3"], np.tile(sb3 / 2, (2, 1)), rtol=0, atol=1e-15)
    for k in ("W1", "b1", "W2", "b2"):
        assert not S[k].any()


def test_mlp_lr_zero_and_empty_batch():
    rng = np.random.default_rng(5)
    p = _mlp_params(rng, 4, 3, 2, 2)
    rows = [[(1, O.f32_bits(2.0))], [(0, O.f32_bits(-1.0)), (3, O.f32_bits(0.5))]]
    new, _ = O.mlp_step(rows, 4, p, [0, 1], 0.0)
    assert all(np.array_equal(new[k], p[k]) for k in p)
    new, g = O.mlp_step([], 4, p, [], 1.0)
    assert all(np.array_equal(new[k], p[k]) and not g[k].any() for k in p)


# --- level order of the live codes -------------------------------------------------
def test_level_order_worked_example(example):
    rows, I, D, N = example
    lo = O.level_order(I, D)
    want = GOLD["level_order"]
    for k in ("order", "parent", "depth", "level_off", "D"):
        assert lo[k] == want[k], k


@pytest.mark.parametrize("seed", range(20))
def test_level_order_invariants_and_decode(seed):
    spec = [dict(n_rows=30, n_cols=9, density=0.8, n_values=2, prefix_copy=0.7),
            dict(n_rows=12, n_cols=25, density=0.4, n_values=3),
            dict(n_rows=60, n_cols=6, density=1.0, n_values=1, prefix_copy=0.5)][seed % 3]
    rp, c, v = tiny_batch(6100 + seed, zeros=(seed % 4 == 0), **spec)
    rows = O.canonicalize(spec["n_rows"], spec["n_cols"], rp, c, v)
    I, D, _ = O.encode(rows)
    lo = O.level_order(I, D)
    cp = O.build_cprime(I, D)
    n = len(lo["order"])
    assert n == O.layout_stats(I, D)["n_live"]
    assert sorted(lo["order"]) == sorted(set(lo["order"]))
    for i, (p, d) in enumerate(zip(lo["parent"], lo["depth"])):
        if d == 1:
            assert p is None
        else:
            assert p < i and lo["depth"][p] == d - 1
            assert lo["order"][p] == cp["parent"][lo["order"][i]]
        if i and lo["depth"][i - 1] == d:
            assert lo["order"][i - 1] < lo["order"][i]          # stable inside a depth
        assert lo["level_off"][d - 1] <= i < lo["level_off"][d]
    assert lo["level_off"][-1] == n and lo["level_off"][0] == 0
    # decoding through the new numbering gives Algorithm 6's rows
    def chain(c):
        out = []
        while c is not None:
            out.append(lo["key"][c])
            c = lo["parent"][c]
        return out[::-1]
    assert [[p for c in d for p in chain(c)] for d in lo["D"]] == O.decode(I, D)
