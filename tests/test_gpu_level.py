"""GPU parity of the device level order (live codes of D and their ancestors,
stably sorted by (depth, index), parents and D renumbered) built from the tree of
toc_cprime_build, with the oracle's level_order on the oracle's unpacking of the
same physical bytes: every array equal, bit for bit; malformed inputs get their
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
PHYS = json.load(open(os.path.join(HERE, "golden", "physical_worked_example.json")))
NONE = 0xFFFFFFFF


def blobs_of(B):
    encs = T.toc_encode_batches(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    return [T.toc_enc_pack(e) for e in encs]


def level_gpu(blobs, max_levels=64, d_counts=None):
    """toc_cprime_build then toc_level_build over the blobs in one launch each;
    returns per batch (parent, col, val bits, depth, level offsets, D) host arrays
    or None where the status is nonzero, and the status array."""
    infos = [T.toc_phys_info_get(b) for b in blobs]
    nb = len(blobs)
    blob_off = np.concatenate([[0], np.cumsum([len(b) for b in blobs])]).astype(np.int64)
    node_off = np.concatenate([[0], np.cumsum([i["n_nodes"] for i in infos])]).astype(np.int64)
    if d_counts is None:
        d_counts = [i["n_codes"] for i in infos]
    d_off = np.concatenate([[0], np.cumsum(d_counts)]).astype(np.int64)
    max_rows = max([i["n_rows"] for i in infos] + [0])
    dblob = torch.from_numpy(np.concatenate([np.asarray(b, np.uint8) for b in blobs]
                                            + [np.zeros(1, np.uint8)])).to(DEV)
    n = int(node_off[-1])
    cp = [torch.empty(n, dtype=torch.int32, device=DEV) for _ in range(4)]
    cst = torch.full((nb,), -1, dtype=torch.int32, device=DEV)
    ws = torch.empty(T.toc_cprime_workspace_size(nb, n), dtype=torch.uint8, device=DEV)
    n_cols = 1 + max([i["max_col"] for i in infos] + [0])
    T.toc_cprime_build(dblob, blob_off, node_off, max_rows, n_cols, cp[0], cp[1], cp[2], cp[3],
                       cst, ws)
    lv = [torch.full((n,), -7, dtype=torch.int32, device=DEV) for _ in range(4)]
    level = torch.full((nb * (max_levels + 1),), -7, dtype=torch.int32, device=DEV)
    lD = torch.full((max(int(d_off[-1]), 1),), -7, dtype=torch.int32, device=DEV)
    counts = torch.full((2 * nb,), -7, dtype=torch.int64, device=DEV)
    st = torch.full((nb,), -1, dtype=torch.int32, device=DEV)
    ws2 = torch.empty(T.toc_level_workspace_size(nb, n), dtype=torch.uint8, device=DEV)
    T.toc_level_build(dblob, blob_off, node_off, d_off, max_levels, cst, cp[0], cp[1], cp[2],
                      cp[3], lv[0], lv[1], lv[2], lv[3], level, lD, counts, st, ws2)
    torch.cuda.synchronize()
    host = [x.cpu().numpy().view(np.uint32) for x in lv]
    level = level.cpu().numpy().view(np.uint32).reshape(nb, max_levels + 1)
    lD = lD.cpu().numpy().view(np.uint32)
    counts, st = counts.cpu().numpy().reshape(nb, 2), st.cpu().numpy()
    per = []
    for b in range(nb):
        if st[b] != 0:
            per.append(None)
            continue
        n_live, top = int(counts[b, 0]), int(counts[b, 1])
        o = int(node_off[b])
        per.append(tuple(h[o:o + n_live] for h in host)
                   + (level[b, :top + 1], lD[d_off[b]:d_off[b + 1]]))
    return per, st


def assert_same(got, blob):
    I, D = O.unpack_physical(bytes(blob))
    lo = O.level_order(I, D)
    parent, col, val, depth, level, lD = got
    assert parent.tolist() == [NONE if p is None else p for p in lo["parent"]]
    assert col.tolist() == [k[0] for k in lo["key"]]
    assert val.tolist() == [k[1] for k in lo["key"]]
    assert depth.tolist() == lo["depth"]
    assert level.tolist() == lo["level_off"]
    assert lD.tolist() == [c for d in lo["D"] for c in d]


def test_worked_example():
    blob = np.frombuffer(bytes.fromhex("".join(a["hex"] for a in PHYS["arrays"])), np.uint8)
    (got,), st = level_gpu([blob])
    assert st.tolist() == [0]
    want = GOLD["level_order"]
    assert got[3].tolist() == want["depth"]
    assert got[4].tolist() == want["level_off"]
    assert got[5].tolist() == [c for d in want["D"] for c in d]
    assert got[0].tolist() == [NONE if p is None else p for p in want["parent"]]
    assert_same(got, blob)


TINY = [dict(n_rows=0, density=0.5, n_values=2),
        dict(n_rows=5, density=0.0, n_values=2),
        dict(n_rows=1, density=1.0, n_values=1),
        dict(n_rows=40, density=0.3, n_values=3, prefix_copy=0.6),
        dict(n_rows=9, density=0.05, n_values=2),
        dict(n_rows=300, density=0.9, n_values=1, prefix_copy=0.9),
        dict(n_rows=250, density=1.0, n_values=2, prefix_copy=0.5)]


def test_tiny_batches_one_launch():
    blobs = []
    for n_cols in (3, 64, 400):
        for i, spec in enumerate(TINY):
            rp, c, v = tiny_batch(800 + i + n_cols, n_cols=n_cols, zeros=(i % 2 == 1), **spec)
            blobs += blobs_of(Batches(n_cols, [spec["n_rows"]], rp, c, v))
    per, st = level_gpu(blobs, max_levels=512)
    assert st.tolist() == [0] * len(blobs)
    for got, blob in zip(per, blobs):
        assert_same(got, blob)


@pytest.mark.parametrize("cfg,first,nb", [("c1", 0, 1), ("c2", 3, 3), ("c3", 5, 2),
                                          ("c4", 0, 1), ("c5", 11, 8)])
def test_config_batches(cfg, first, nb):
    blobs = blobs_of(config_batches(cfg, first, nb))
    per, st = level_gpu(blobs)
    assert st.tolist() == [0] * nb
    for got, blob in zip(per, blobs):
        assert_same(got, blob)


def test_statuses():
    """A batch deeper than max_levels, a d_off span that is not the blob's |D| and
    a blob cut short: each gets its status, the good batches their level order."""
    good = blobs_of(config_batches("c5", 0, 2))
    deep = blobs_of(config_batches("c1", 0, 1))               # depth 41 > 8
    bad = np.asarray(good[0][:-3], np.uint8)                  # malformed: cprime rejects it
    blobs = [good[0], deep[0], good[1], bad]
    d_counts = [T.toc_phys_info_get(b)["n_codes"] for b in blobs[:3]] + [0]
    # the malformed blob has no |D| of its own: give it 0 entries
    per, st = level_gpu_checked(blobs, d_counts)
    assert st[0] == 0 and st[2] == 0
    assert st[1] == T.TOC_LEVEL_DEPTH
    assert st[3] == T.TOC_CPRIME_LAYOUT
    assert_same(per[0], good[0])
    assert_same(per[2], good[1])
    # |D| of batch 1 declared one short
    d2 = [T.toc_phys_info_get(b)["n_codes"] for b in good]
    per, st = level_gpu(good, d_counts=[d2[0], d2[1] - 1])
    assert st.tolist() == [0, T.TOC_LEVEL_D]
    assert_same(per[0], good[0])


def level_gpu_checked(blobs, d_counts):
    """level_gpu for a list holding a malformed last blob: its node count is taken
    as 1 (the cprime status marks it; nothing of its range is read)."""
    real_info = T.toc_phys_info_get
    def info(b):
        try:
            return real_info(b)
        except T.TocError:
            return {"n_nodes": 1, "n_rows": 0, "n_codes": 0, "max_col": -1}
    T.toc_phys_info_get = info
    try:
        return level_gpu(blobs, max_levels=8, d_counts=d_counts)
    finally:
        T.toc_phys_info_get = real_info


def ingest_right(blobs, w_host, max_levels=64, cprime_n_cols=None, cprime_status=None):
    """Physical bytes -> toc_cprime_build -> toc_level_build -> toc_level_right_mul,
    all on the device; returns R (host, one value per row) and the statuses.
    cprime_n_cols: n_cols of the C' build (default: one past the largest column);
    cprime_status: a list that receives the C' build's statuses."""
    infos = [T.toc_phys_info_get(b) for b in blobs]
    nb = len(blobs)
    blob_off = np.concatenate([[0], np.cumsum([len(b) for b in blobs])]).astype(np.int64)
    node_off = np.concatenate([[0], np.cumsum([i["n_nodes"] for i in infos])]).astype(np.int64)
    d_off = np.concatenate([[0], np.cumsum([i["n_codes"] for i in infos])]).astype(np.int64)
    row_off = np.concatenate([[0], np.cumsum([i["n_rows"] for i in infos])]).astype(np.int64)
    max_rows = max([i["n_rows"] for i in infos] + [0])
    dblob = torch.from_numpy(np.concatenate([np.asarray(b, np.uint8) for b in blobs]
                                            + [np.zeros(1, np.uint8)])).to(DEV)
    n = int(node_off[-1])
    cp = [torch.empty(n, dtype=torch.int32, device=DEV) for _ in range(4)]
    cst = torch.empty(nb, dtype=torch.int32, device=DEV)
    ws = torch.empty(T.toc_cprime_workspace_size(nb, n), dtype=torch.uint8, device=DEV)
    n_cols = 1 + max([i["max_col"] for i in infos] + [0]) if cprime_n_cols is None \
        else cprime_n_cols
    T.toc_cprime_build(dblob, blob_off, node_off, max_rows, n_cols, *cp, cst, ws)
    lv = [torch.empty(n, dtype=torch.int32, device=DEV) for _ in range(4)]
    level = torch.empty(nb * (max_levels + 1), dtype=torch.int32, device=DEV)
    lD = torch.empty(max(int(d_off[-1]), 1), dtype=torch.int32, device=DEV)
    counts = torch.empty(2 * nb, dtype=torch.int64, device=DEV)
    lst = torch.empty(nb, dtype=torch.int32, device=DEV)
    ws2 = torch.empty(T.toc_level_workspace_size(nb, n), dtype=torch.uint8, device=DEV)
    T.toc_level_build(dblob, blob_off, node_off, d_off, max_levels, cst, *cp, *lv, level, lD,
                      counts, lst, ws2)
    max_live = int(counts.view(-1, 2)[:, 0].max().item())
    wd = torch.from_numpy(np.asarray(w_host, np.float32)).to(DEV)
    r = torch.full((max(int(row_off[-1]), 1),), float("nan"), device=DEV)
    st = torch.full((nb,), -1, dtype=torch.int32, device=DEV)
    ws3 = torch.empty(32 * (nb + 1), dtype=torch.uint8, device=DEV)
    T.toc_level_right_mul(dblob, blob_off, node_off, d_off, row_off, max_levels, max_live, lst,
                          counts, level, lv[0], lv[1], lv[2], lD, wd, r, st, ws3)
    torch.cuda.synchronize()
    if cprime_status is not None:
        cprime_status.extend(cst.cpu().numpy().tolist())
    return r.cpu().numpy()[:int(row_off[-1])], st.cpu().numpy(), row_off


@pytest.mark.parametrize("cfg,first,nb", [("c1", 0, 1), ("c2", 3, 3), ("c3", 5, 2), ("c5", 11, 8)])
def test_ingest_right_product(cfg, first, nb):
    """A.w from physical bytes entirely on the device, within 1e-5 S of the oracle's
    fp64 product on the decoded batch."""
    from workloads import config_W
    B = config_batches(cfg, first, nb)
    blobs = blobs_of(B)
    w = config_W(cfg, 1)[:, 0]
    r, st, row_off = ingest_right(blobs, w)
    assert st.tolist() == [0] * nb
    for b in range(nb):
        n, rp, c, v = B.batch(b)
        rows = O.canonicalize(n, B.n_cols, rp, c, v)
        want, S = O.dense_right(rows, B.n_cols, w[:, None].astype(np.float64))
        got = r[row_off[b]:row_off[b + 1]]
        assert np.all(np.abs(got - want[:, 0]) <= 1e-5 * S[:, 0]), f"batch {b}"


def test_ingest_right_tiny_and_empty():
    blobs = []
    for i, spec in enumerate(TINY):
        rp, c, v = tiny_batch(900 + i, n_cols=64, zeros=(i % 2 == 0), **spec)
        blobs += blobs_of(Batches(64, [spec["n_rows"]], rp, c, v))
    w = np.random.default_rng(3).standard_normal(64).astype(np.float32)
    r, st, row_off = ingest_right(blobs, w, max_levels=512)
    assert st.tolist() == [0] * len(blobs)
    for b, blob in enumerate(blobs):
        I, D = O.unpack_physical(bytes(blob))
        rows = O.decode(I, D)
        want, S = O.dense_right(rows, 64, w[:, None].astype(np.float64))
        got = r[row_off[b]:row_off[b + 1]]
        assert np.all(np.abs(got - want[:, 0]) <= 1e-5 * S[:, 0]), f"batch {b}"


def test_columns_past_n_cols():
    """Batch 1 uses columns up to 63, batch 0 only columns below 32.  Built for 32
    columns, batch 1's bytes are malformed (TOC_CPRIME_COLUMN from the C' build,
    carried through the level order and the product) while batch 0 is built and
    multiplied as usual.  Built for 64 columns but multiplied by a w of 32 entries,
    the product reports TOC_CPRIME_COLUMN for batch 1 and never reads w past its
    end; batch 0 is unaffected."""
    rp0, c0, v0 = tiny_batch(5, n_rows=20, n_cols=32, density=0.5, n_values=3, prefix_copy=0.5)
    rp1, c1, v1 = tiny_batch(6, n_rows=20, n_cols=64, density=0.5, n_values=3, prefix_copy=0.5)
    blobs = blobs_of(Batches(32, [20], rp0, c0, v0)) + blobs_of(Batches(64, [20], rp1, c1, v1))
    assert T.toc_phys_info_get(blobs[0])["max_col"] < 32 <= T.toc_phys_info_get(blobs[1])["max_col"]
    w = np.random.default_rng(8).standard_normal(32).astype(np.float32)
    rows0 = O.canonicalize(20, 32, rp0, c0, v0)
    want, S = O.dense_right(rows0, 32, w[:, None].astype(np.float64))
    for n_cols, want_cp in ((32, [0, T.TOC_CPRIME_COLUMN]), (64, [0, 0])):
        cst = []
        r, st, row_off = ingest_right(blobs, w, cprime_n_cols=n_cols, cprime_status=cst)
        assert cst == want_cp
        assert st.tolist() == [0, T.TOC_CPRIME_COLUMN]
        assert np.all(np.abs(r[:20] - want[:, 0]) <= 1e-5 * S[:, 0])
        assert np.all(np.isnan(r[20:40]))           # batch 1's rows are not written
