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
