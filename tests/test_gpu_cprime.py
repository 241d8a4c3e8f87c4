"""GPU parity of the device-side decoding tree (Algorithm 2, section 4.1.2) built
from the physical encoding (section 3.2) with the oracle's build_cprime on the
oracle's unpacking of the same bytes, node by node and bit for bit; malformed
blobs get their status code without disturbing the other batches of a launch."""

import json
import os

import numpy as np
import pytest

import oracle as O
import paper_1702_06943_amd as T
from workloads import config_batches, tiny_batch, Batches

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"
HERE = os.path.dirname(os.path.abspath(__file__))
GOLD = json.load(open(os.path.join(HERE, "golden", "worked_example.json")))
PHYS = json.load(open(os.path.join(HERE, "golden", "physical_worked_example.json")))
NONE = 0xFFFFFFFF


def blobs_of(B):
    encs = T.toc_encode_batches(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    return [T.toc_enc_pack(e) for e in encs]


def build_gpu(blobs, n_nodes=None, max_rows=None, n_cols=None):
    """Runs toc_cprime_build over the blobs in one launch; returns per-batch
    (parent, col, val bits, depth) host arrays and the status array.  n_cols
    defaults to one past the largest column of any blob's I."""
    if n_nodes is None:
        n_nodes = [T.toc_phys_info_get(b)["n_nodes"] for b in blobs]
    if max_rows is None:
        max_rows = max([T.toc_phys_info_get(b)["n_rows"] for b in blobs] + [0])
    if n_cols is None:
        n_cols = 1 + max([T.toc_phys_info_get(b)["max_col"] for b in blobs] + [0])
    blob_off = np.concatenate([[0], np.cumsum([len(b) for b in blobs])]).astype(np.int64)
    node_off = np.concatenate([[0], np.cumsum(n_nodes)]).astype(np.int64)
    cat = np.concatenate([np.asarray(b, np.uint8) for b in blobs] + [np.zeros(1, np.uint8)])
    dblob = torch.from_numpy(cat).to(DEV)
    n = int(node_off[-1])
    outs = [torch.full((n,), -7, dtype=torch.int32, device=DEV) for _ in range(4)]
    status = torch.full((len(blobs),), -1, dtype=torch.int32, device=DEV)
    ws = torch.empty(T.toc_cprime_workspace_size(len(blobs), n), dtype=torch.uint8, device=DEV)
    T.toc_cprime_build(dblob, blob_off, node_off, max_rows, n_cols, outs[0], outs[1], outs[2],
                       outs[3], status, ws)
    torch.cuda.synchronize()
    host = [o.cpu().numpy().view(np.uint32) for o in outs]
    per = [tuple(h[node_off[b]:node_off[b + 1]] for h in host) for b in range(len(blobs))]
    return per, status.cpu().numpy()


def oracle_arrays(blob):
    I, D = O.unpack_physical(bytes(blob))
    cp = O.build_cprime(I, D)
    parent = np.array([NONE] + cp["parent"][1:], np.uint32)
    col = np.array([NONE] + [k[0] for k in cp["key"][1:]], np.uint32)
    val = np.array([0] + [k[1] for k in cp["key"][1:]], np.uint32)
    depth = np.array(cp["depth"], np.uint32)
    return parent, col, val, depth


def assert_same(got, blob):
    want = oracle_arrays(blob)
    for name, g, w in zip(("parent", "col", "val", "depth"), got, want):
        assert np.array_equal(g, w), f"{name} differs at {np.flatnonzero(g != w)[:5]}"


def test_worked_example_table4():
    blob = np.frombuffer(bytes.fromhex("".join(a["hex"] for a in PHYS["arrays"])), np.uint8)
    (got,), status = build_gpu([blob])
    assert status.tolist() == [0]
    parent, col, val, depth = got
    cp = GOLD["cprime"]
    assert parent[1:].tolist() == cp["parent"][1:]
    assert col[1:].tolist() == [k[0] for k in cp["key"][1:]]
    assert val[1:].tolist() == [O.f32_bits(k[1]) for k in cp["key"][1:]]
    assert depth.tolist() == [0, 1, 1, 1, 1, 1, 2, 2, 2, 3, 2]
    assert_same(got, blob)


TINY = [dict(n_rows=0, density=0.5, n_values=2),
        dict(n_rows=5, density=0.0, n_values=2),
        dict(n_rows=1, density=1.0, n_values=1),
        dict(n_rows=40, density=0.3, n_values=3, prefix_copy=0.6),
        dict(n_rows=9, density=0.05, n_values=2),
        dict(n_rows=300, density=0.9, n_values=1, prefix_copy=0.9)]


def test_tiny_batches_one_launch():
    blobs = []
    for n_cols in (3, 64, 1000):
        for i, spec in enumerate(TINY):
            rp, c, v = tiny_batch(500 + i + n_cols, n_cols=n_cols, **spec)
            blobs += blobs_of(Batches(n_cols, [spec["n_rows"]], rp, c, v))
    per, status = build_gpu(blobs)
    assert status.tolist() == [0] * len(blobs)
    for got, blob in zip(per, blobs):
        assert_same(got, blob)


@pytest.mark.parametrize("cfg,first,nb", [("c1", 0, 1), ("c2", 3, 3), ("c3", 7, 4), ("c4", 1, 1),
                                          ("c5", 11, 6)])
def test_config_batches(cfg, first, nb):
    blobs = blobs_of(config_batches(cfg, first, nb))
    per, status = build_gpu(blobs)
    assert status.tolist() == [0] * nb
    for got, blob in zip(per, blobs):
        assert_same(got, blob)


def test_many_batches_sampled():
    """400 c3 batches in one launch: sampled batches against the oracle, every batch
    against invariants that hold at any size (parent below the node, depth one more
    than the parent's, first layer under the root)."""
    B = config_batches("c3", 100, 400)
    blobs = blobs_of(B)
    per, status = build_gpu(blobs)
    assert np.all(status == 0)
    for b in (0, 137, 399):
        assert_same(per[b], blobs[b])
    for (parent, col, val, depth), blob in zip(per, blobs):
        nI = T.toc_phys_info_get(blob)["n_first"]
        idx = np.arange(len(parent))
        assert np.all(parent[1:nI + 1] == 0) and np.all(depth[1:nI + 1] == 1)
        new = idx[nI + 1:]
        assert np.all(parent[new] < new) and np.all(parent[new] >= 1)
        assert np.array_equal(depth[new], depth[parent[new]] + 1)
        assert np.all(col[1:] < 784)


def _example():
    return bytearray(bytes.fromhex("".join(a["hex"] for a in PHYS["arrays"])))


def test_malformed_blobs_get_status():
    """Planted mistakes in copies of the worked example's bytes, between good
    batches of the same launch (offsets: I columns at 5, values at 15, value
    indexes at 36, D codes at 46, tuple starts at 60)."""
    good = blobs_of(config_batches("c5", 2, 2))
    ex = _example()

    def mut(*pv):
        b = bytearray(ex)
        for pos, v in zip(pv[::2], pv[1::2]):
            b[pos] = v
        return np.frombuffer(bytes(b), np.uint8)

    cases = [
        (mut(36, 4), 11, T.TOC_CPRIME_VALUE_INDEX),   # value index 4 of 4 unique values
        (mut(46, 0), 11, T.TOC_CPRIME_CODE),          # code 0 (the root)
        (mut(50, 9), 11, T.TOC_CPRIME_CODE),          # tuple 2 names node 9 before it exists
        (mut(62, 8, 63, 6), 11, T.TOC_CPRIME_STARTS), # tuple starts 0,4,8,6,9
        (np.frombuffer(bytes(ex), np.uint8), 12, T.TOC_CPRIME_NODES),
        (np.frombuffer(bytes(ex[:-2]), np.uint8), 11, T.TOC_CPRIME_LAYOUT),
        (mut(4, 5), 11, T.TOC_CPRIME_LAYOUT),         # 5 bytes per integer
    ]
    blobs = [good[0]] + [c[0] for c in cases] + [good[1]]
    n_nodes = [T.toc_phys_info_get(good[0])["n_nodes"]] + [c[1] for c in cases] + \
        [T.toc_phys_info_get(good[1])["n_nodes"]]
    per, status = build_gpu(blobs, n_nodes=n_nodes, max_rows=250, n_cols=900)
    assert status.tolist() == [0] + [c[2] for c in cases] + [0]
    assert_same(per[0], good[0])
    assert_same(per[-1], good[1])


def test_column_past_n_cols_gets_status():
    """The worked example's bytes with the third column of I raised from 2 to 4 (a
    column past the 4 of the matrix): TOC_CPRIME_COLUMN, while the unchanged copy
    before it in the same launch is built as usual."""
    ex = _example()
    assert ex[7] == 2
    bad = bytearray(ex)
    bad[7] = 4
    blobs = [np.frombuffer(bytes(ex), np.uint8), np.frombuffer(bytes(bad), np.uint8)]
    assert T.toc_phys_info_get(blobs[1])["max_col"] == 4
    per, status = build_gpu(blobs, n_nodes=[11, 11], max_rows=4, n_cols=4)
    assert status.tolist() == [0, T.TOC_CPRIME_COLUMN]
    assert_same(per[0], blobs[0])


def test_rows_beyond_max_rows():
    ex = np.frombuffer(bytes(_example()), np.uint8)
    (_, ), status = build_gpu([ex], n_nodes=[11], max_rows=3)
    assert status.tolist() == [T.TOC_CPRIME_ROWS]
