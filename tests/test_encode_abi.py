"""CPU tests of the C ABI's host half: symbols, encoder parity with the oracle
(bit-exact I and D), sizes, error paths.  No GPU call is made."""

import json
import os
import re

import numpy as np
import pytest

import oracle as O
import paper_1702_06943_amd as T
from workloads import CONFIGS, config_batches, tiny_batch

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
GOLD = json.load(open(os.path.join(HERE, "golden", "worked_example.json")))


def test_library_exports_every_declared_symbol():
    header = open(os.path.join(ROOT, "include", "toc.h")).read()
    names = set(re.findall(r"\b(toc_[a-z_]+)\s*\(", header))
    assert {"toc_encode", "toc_upload", "toc_right_mul", "toc_left_mul",
            "toc_decode_csr"} <= names
    lib = T.lib()
    for n in sorted(names):
        assert hasattr(lib, n), n


def _oracle_encode(n_rows, n_cols, rp, c, v):
    rows = O.canonicalize(n_rows, n_cols, rp, c, v)
    I, D, N = O.encode(rows)
    return rows, I, D, N


def _assert_same_encoding(enc, I, D, N):
    I_col, I_val, D_rp, D_codes = T.toc_enc_export(enc)
    assert [(int(c), int(b)) for c, b in zip(I_col, I_val.view(np.uint32))] == I
    flat = [x for d in D for x in d]
    assert D_codes.tolist() == flat
    assert D_rp.tolist() == list(np.cumsum([0] + [len(d) for d in D]))
    assert T.toc_enc_info_get(enc)["n_nodes"] == N


def test_worked_example_encoding():
    rows_in = GOLD["rows_from_table2"]["rows"]
    rp = np.cumsum([0] + [len(r) for r in rows_in])
    c = np.array([p[0] for r in rows_in for p in r], np.int32)
    v = np.array([p[1] for r in rows_in for p in r], np.float32)
    enc = T.toc_encode(4, 4, rp, c, v)
    I_col, I_val, D_rp, D_codes = T.toc_enc_export(enc)
    assert I_col.tolist() == [p[0] for p in GOLD["I"]["pairs"]]
    assert np.array_equal(I_val, np.array([p[1] for p in GOLD["I"]["pairs"]], np.float32))
    assert D_codes.tolist() == [x for d in GOLD["D"]["codes"] for x in d]
    info = T.toc_enc_info_get(enc)
    s = GOLD["sizes"]
    assert (info["n_live"], info["n_deep"], info["max_depth"], info["n_nodes"],
            info["canon_bytes"], info["phys_bytes"]) == (
        s["n_live"], s["n_deep"], s["max_depth"], s["n_nodes"], s["canon_bytes"],
        s["physical_bytes"])


TINY = [
    dict(n_rows=1, n_cols=1, density=1.0, n_values=1),
    dict(n_rows=9, n_cols=7, density=0.8, n_values=2, prefix_copy=0.6),
    dict(n_rows=25, n_cols=12, density=0.9, n_values=2, prefix_copy=0.9),
    dict(n_rows=40, n_cols=30, density=0.3, n_values=5),
    dict(n_rows=16, n_cols=5, density=1.0, n_values=1),
]


@pytest.mark.parametrize("seed", range(15))
@pytest.mark.parametrize("case", range(len(TINY)))
def test_encoder_bit_exact_vs_oracle_tiny(seed, case):
    spec = TINY[case]
    rp, c, v = tiny_batch(5000 + seed * 17 + case, zeros=(seed % 3 == 0), **spec)
    rows, I, D, N = _oracle_encode(spec["n_rows"], spec["n_cols"], rp, c, v)
    enc = T.toc_encode(spec["n_rows"], spec["n_cols"], rp, c, v)
    _assert_same_encoding(enc, I, D, N)
    info = T.toc_enc_info_get(enc)
    st = O.layout_stats(I, D)
    for key in ("n_live", "n_deep", "max_depth", "canon_bytes", "n_codes", "n_first"):
        assert info[key] == st[key], key
    assert info["phys_bytes"] == O.physical_bytes(I, D)
    assert info["nnz"] == sum(len(r) for r in rows)


@pytest.mark.parametrize("cfg", sorted(CONFIGS))
def test_encoder_bit_exact_vs_oracle_configs(cfg):
    B = config_batches(cfg, 3 if CONFIGS[cfg]["n_batches"] > 3 else 0, 1)
    n, rp, c, v = B.batch(0)
    rows, I, D, N = _oracle_encode(n, B.n_cols, rp, c, v)
    enc = T.toc_encode(n, B.n_cols, rp, c, v)
    _assert_same_encoding(enc, I, D, N)
    info = T.toc_enc_info_get(enc)
    st = O.layout_stats(I, D)
    assert info["canon_bytes"] == st["canon_bytes"]
    assert info["n_live"] == st["n_live"]


def test_encode_batches_matches_single():
    B = config_batches("c5", 0, 6)
    encs = T.toc_encode_batches(B.n_rows, B.n_cols, B.rowptr, B.col, B.val, n_threads=3)
    for b in range(B.n_batches):
        n, rp, c, v = B.batch(b)
        one = T.toc_encode(n, B.n_cols, rp, c, v)
        for x, y in zip(T.toc_enc_export(encs[b]), T.toc_enc_export(one)):
            assert np.array_equal(x, y)


def test_empty_and_all_zero_batches():
    e = T.toc_encode(0, 3, [0], [], np.zeros(0, np.float32))
    info = T.toc_enc_info_get(e)
    assert info["n_nodes"] == 1 and info["n_codes"] == 0 and info["canon_bytes"] == 8
    e = T.toc_encode(3, 4, [0, 2, 2, 3], [0, 3, 1],
                     np.array([0.0, -0.0, 0.0], np.float32))
    info = T.toc_enc_info_get(e)
    assert (info["nnz"], info["n_first"], info["n_codes"], info["n_nodes"]) == (0, 0, 0, 1)


@pytest.mark.parametrize("bad", [
    dict(n_rows=1, rowptr=[0, 2], col=[1, 1], val=[1, 2]),
    dict(n_rows=1, rowptr=[0, 2], col=[2, 1], val=[1, 2]),
    dict(n_rows=1, rowptr=[0, 1], col=[4], val=[1]),
    dict(n_rows=1, rowptr=[0, 1], col=[-1], val=[1]),
    dict(n_rows=1, rowptr=[0, 1], col=[0], val=[np.nan]),
    dict(n_rows=1, rowptr=[0, 1], col=[0], val=[-np.inf]),
    dict(n_rows=1, rowptr=[1, 1], col=[0], val=[1]),
    dict(n_rows=2, rowptr=[0, 2, 1], col=[0, 1], val=[1, 1]),
    dict(n_rows=-1, rowptr=[0], col=[], val=[]),
])
def test_encode_rejects(bad):
    with pytest.raises(T.TocError) as ei:
        T.toc_encode(bad["n_rows"], 4, bad["rowptr"], bad["col"],
                     np.array(bad["val"], np.float32))
    assert ei.value.status == T.TOC_EINVAL


def test_encode_batches_error_frees_everything():
    rp = np.array([0, 1, 2], np.int64)
    with pytest.raises(T.TocError) as ei:
        T.toc_encode_batches([1, 1], 4, rp, np.array([0, 9], np.int32),
                             np.ones(2, np.float32))
    assert ei.value.status == T.TOC_EINVAL and "batch 1" in str(ei.value)


def test_null_pointers_rejected():
    lib = T.lib()
    assert lib.toc_encode(1, 1, None, None, None, None) == T.TOC_EINVAL
    assert lib.toc_enc_info_get(None, None) == T.TOC_EINVAL
    assert lib.toc_upload_size(None, 1, 0, None) == T.TOC_EINVAL
    assert lib.toc_right_mul(None, None, 1, 1, None, 1, None, 0, None) == T.TOC_EINVAL
    assert lib.toc_left_mul(None, None, 1, 1, None, 1, 0, None, 0, None) == T.TOC_EINVAL
    assert lib.toc_decode_csr(None, None, None, None, None) == T.TOC_EINVAL
    assert lib.toc_map_values(None, 0, 1.0, None) == T.TOC_EINVAL
    assert lib.toc_decode_dense(None, 0.0, None, 1, None) == T.TOC_EINVAL


@pytest.mark.parametrize("seed", range(6))
def test_bench_variant_sizes_match_oracle(seed):
    """The benchmark's ablation sizes (section 5.2), computed from the encoder's
    counts, equal the oracle's dense_bytes / sparse_bytes / logical_bytes /
    physical_bytes on the same batches."""
    import bench
    infos, want = [], {"dense": 0, "sparse": 0, "logical": 0, "full": 0}
    for k, spec in enumerate(TINY):
        rp, c, v = tiny_batch(8800 + 7 * seed + k, zeros=(seed % 2 == 0), **spec)
        rows, I, D, N = _oracle_encode(spec["n_rows"], spec["n_cols"], rp, c, v)
        enc = T.toc_encode(spec["n_rows"], 40, rp, c, v)
        infos.append(T.toc_enc_info_get(enc))
        want["dense"] += O.dense_bytes(spec["n_rows"], 40)
        want["sparse"] += O.sparse_bytes(rows)
        want["logical"] += O.logical_bytes(I, D)
        want["full"] += O.physical_bytes(I, D)
    got = bench.variant_sizes(infos, 40)
    for key, val in want.items():
        assert got[f"{key}_bytes"] == val, key


def test_encode_device_host_checks():
    """Argument checks of the device encoder that return before any HIP call."""
    import ctypes as C
    lib = T.lib()
    n = C.c_size_t()
    assert lib.toc_encode_device_workspace_size(-1, 10, C.byref(n)) == T.TOC_EINVAL
    assert lib.toc_encode_device_workspace_size(3, (1 << 30) + 1, C.byref(n)) == \
        T.TOC_EUNSUPPORTED
    assert lib.toc_encode_device_workspace_size(0, 100, C.byref(n)) == 0 and n.value == 0
    assert lib.toc_encode_device_workspace_size(2, 1000, C.byref(n)) == 0
    small = n.value
    assert lib.toc_encode_device_workspace_size(2, 100000, C.byref(n)) == 0 and n.value > small
    nr = np.array([3, 2], np.int32)
    dummy = C.c_void_p(16)                     # never dereferenced: every check fails first
    args = [2, nr.ctypes.data, 5, dummy, dummy, dummy, 10, 6, dummy, dummy, dummy, dummy,
            dummy, dummy, dummy, 1, None]
    assert lib.toc_encode_device(*args) == T.TOC_ESIZE          # workspace of 1 byte
    bad = list(args)
    bad[0] = -1
    assert lib.toc_encode_device(*bad) == T.TOC_EINVAL
    bad = list(args)
    bad[7] = (1 << 30) + 1
    assert lib.toc_encode_device(*bad) == T.TOC_EUNSUPPORTED
    bad = list(args)
    bad[3] = None
    assert lib.toc_encode_device(*bad) == T.TOC_EINVAL
    nr_bad = np.array([3, -2], np.int32)
    bad = list(args)
    bad[1] = nr_bad.ctypes.data
    assert lib.toc_encode_device(*bad) == T.TOC_EINVAL
    assert lib.toc_encode_device(0, None, 5, None, None, None, 0, 0, None, None, None, None,
                                 None, None, None, 0, None) == 0
