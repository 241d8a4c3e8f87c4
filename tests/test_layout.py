"""CPU checks of the upload image (TOC_UPLOAD_HOST writes it into host memory).

The image is read back with numpy and checked against the invariants of the
decoding tree (Algorithm 2) and against the oracle: walking it must decode every
batch exactly and give the same fp64 products.
"""

import numpy as np
import pytest

import oracle as O
import paper_1702_06943_amd as T
from workloads import config_batches, tiny_batch


def read_image(dev, buf):
    L = T.toc_dev_layout_get(dev)
    info = T.toc_dev_info_get(dev)
    nb = info["n_batches"]
    bt = np.frombuffer(buf, T.BATCH_DTYPE, count=nb, offset=L["batches"])

    def arr(name, dtype, count):
        return np.frombuffer(buf, dtype, count=count, offset=L[name])

    n_codes = info["n_stored"]
    n_levels = int((bt["n_levels"] + 1).sum()) if nb else 0
    img = dict(
        bt=bt, info=info,
        level=arr("level", np.uint32, n_levels),
        key=arr("key", T.KEY_DTYPE, n_codes),
        link=arr("link", T.LINK_DTYPE, info["n_deep"]),
        span=arr("span", np.uint32, int((bt["n_rows"] + 1).sum()) if nb else 0),
        dcodes=arr("dcodes", np.uint32, info["n_codes"]),
        occ_off=arr("occ_off", np.uint32, n_codes + 2 * nb),
        tlist=arr("tlist", np.uint32,
                  int((bt["n_int1"] + bt["n_codes"] - bt["n_lvl1"]).sum()) if nb else 0),
        cols=arr("cols", np.uint32, nb * 4 * (info["n_cols"] + 1)),
        tchild=arr("tchild", np.uint32,
                   int((bt["n_int1"] + bt["n_codes"] - bt["n_lvl1"] + 1).sum()) if nb else 0),
        centry=arr("centry", np.uint32, info["n_codes"] + (
            int((bt["n_int1"] + bt["n_codes"] - bt["n_lvl1"]).sum()) if nb else 0)),
        cval=arr("cval", np.float32, info["n_codes"] + (
            int((bt["n_int1"] + bt["n_codes"] - bt["n_lvl1"]).sum()) if nb else 0)),
    )
    for f in ("col", "val"):
        img[f] = img["key"][f]
    return img


def batch_view(img, b):
    t = img["bt"][b]
    m = int(img["info"]["n_cols"])
    cb, nc = int(t["code_base"]), int(t["n_codes"])
    # links are stored for the codes of depth >= 2 only; a depth-1 code has no
    # parent and depth 1
    n1, db = int(t["n_lvl1"]), int(t["deep_base"])
    parent = np.full(nc, 0xFFFFFFFF, np.uint32)
    depth = np.ones(nc, np.uint32)
    parent[n1:] = img["link"]["parent"][db:db + nc - n1]
    depth[n1:] = img["link"]["depth"][db:db + nc - n1]
    return dict(
        t=t,
        level=img["level"][int(t["lvl_base"]):int(t["lvl_base"]) + int(t["n_levels"]) + 1],
        parent=parent, col=img["col"][cb:cb + nc],
        val=img["val"][cb:cb + nc], depth=depth,
        span=img["span"][int(t["span_base"]):int(t["span_base"]) + int(t["n_rows"]) + 1],
        dc=img["dcodes"][int(t["d_base"]):int(t["d_base"]) + int(t["n_d"])],
        occ_off=img["occ_off"][cb + 2 * b:cb + 2 * b + nc + 2],
        tlist=img["tlist"][int(t["tree_base"]):int(t["tree_base"]) + int(t["n_int1"]) + nc
                           - int(t["n_lvl1"])],
        cols=img["cols"][b * 4 * (m + 1):(b + 1) * 4 * (m + 1)].reshape(4, m + 1),
        tchild=img["tchild"][int(t["tree_base"]) + b:int(t["tree_base"]) + b + int(t["n_int1"]) + nc
                             - int(t["n_lvl1"]) + 1],
        centry=img["centry"][int(t["d_base"]) + int(t["tree_base"]):
                             int(t["d_base"]) + int(t["tree_base"]) + int(t["n_d"]) + int(t["n_int1"])
                             + nc - int(t["n_lvl1"])],
        cval=img["cval"][int(t["d_base"]) + int(t["tree_base"]):
                         int(t["d_base"]) + int(t["tree_base"]) + int(t["n_d"]) + int(t["n_int1"])
                         + nc - int(t["n_lvl1"])],
    )


def check_invariants(v):
    t = v["t"]
    nc, n1, ni, nl = int(t["n_codes"]), int(t["n_lvl1"]), int(t["n_int1"]), int(t["n_levels"])
    lv = v["level"]
    assert lv[0] == 0 and lv[-1] == nc and np.all(np.diff(lv.astype(np.int64)) >= 0)
    assert (lv[1] if nl else 0) == n1
    for d in range(1, nl + 1):
        codes = np.arange(lv[d - 1], lv[d])
        assert np.all(v["depth"][codes] == d)
        if d == 1:
            assert np.all(v["parent"][codes] == 0xFFFFFFFF)
        else:
            p = v["parent"][codes]
            assert np.all((p >= lv[d - 2]) & (p < lv[d - 1])), "parent one level up"
    # depth-1 codes with children come first
    has_child = np.zeros(nc, bool)
    deep = v["parent"] != 0xFFFFFFFF
    has_child[v["parent"][deep]] = True
    assert np.all(has_child[:ni]) and not np.any(has_child[ni:n1])
    # siblings have distinct keys
    keys = set()
    for c in range(nc):
        k = (int(v["parent"][c]), int(v["col"][c]), int(v["val"][c:c + 1].view(np.uint32)[0]))
        assert k not in keys
        keys.add(k)
    assert np.all(v["dc"] < nc)
    assert v["span"][0] == 0 and v["span"][-1] == len(v["dc"])
    # depth-1 leaves numbered by their first entry in D; deeper levels sorted by
    # parent
    first_entry = {}
    for j, c in enumerate(v["dc"].tolist()):
        first_entry.setdefault(c, j)
    fe = [first_entry[c] for c in range(ni, n1)]
    assert fe == sorted(fe)
    for d in range(2, nl + 1):
        assert np.all(np.diff(v["parent"][lv[d - 1]:lv[d]].astype(np.int64)) >= 0)
    # left positions: leaves ordered by (column, code) after the codes with
    # children; every other code at its own index
    at = list(range(ni)) + sorted(range(ni, n1), key=lambda c: (int(v["col"][c]), c)) \
        + list(range(n1, nc))
    # the tuples holding each position's code (the index set of the sum that
    # defines G(x) in Theorem 2), ascending
    row_of = np.repeat(np.arange(len(v["span"]) - 1), np.diff(v["span"].astype(np.int64)))
    occ = [row_of[v["dc"] == at[p]] for p in range(nc)]
    bits = v["val"].view(np.uint32)
    # tree list: codes with children or depth >= 2, sorted by column
    tree = [c for c in range(nc) if c < ni or c >= n1]
    tl = v["tlist"]
    assert sorted(tl.tolist()) == tree
    assert np.all(np.diff(v["col"][tl].astype(np.int64)) >= 0)
    # the entries of the left multiplication, in three parts, with the value of
    # the entry's code beside each (0 in the third part)
    ce, cvb = v["centry"], v["cval"].view(np.uint32)
    oo = v["occ_off"]
    lo, to = oo[:n1 - ni + 1], oo[n1 - ni + 1:]
    assert len(to) == len(tree) + 1
    o = 0
    for p in range(ni, n1):           # 1: leaf occurrences by position, bit 31 on the first
        k = len(occ[p])
        assert lo[p - ni] == o
        assert np.array_equal(ce[o:o + k] & 0x7FFFFFFF, occ[p])
        assert k == 0 or (ce[o] >> 31 == 1 and np.all(ce[o + 1:o + k] >> 31 == 0))
        assert np.all(cvb[o:o + k] == bits[at[p]])
        o += k
    assert lo[n1 - ni] == o
    n_lo = o
    assert np.array_equal(ce[o:o + len(tl)], tl | np.uint32(0x40000000))   # 2: tree codes
    assert np.array_equal(cvb[o:o + len(tl)], bits[tl])
    o += len(tl)
    for h, c in enumerate(tree):      # 3: the tree codes' tuples, by tree row
        k = len(occ[c])
        assert to[h] == o
        assert np.array_equal(ce[o:o + k], occ[c]) and not cvb[o:o + k].any()
        o += k
    assert to[len(tree)] == o == len(v["dc"]) + len(tree) == len(ce)
    # column index: first leaf position, leaf occurrences before it and first
    # tree-list entry of each column j; columns by entry count, most first (ties
    # by column)
    cx = v["cols"]
    m = cx.shape[1] - 1
    leaf_cols = v["col"][ni:n1].astype(np.int64)
    tree_cols = v["col"][tl].astype(np.int64)
    for j in range(m + 1):
        lc = ni + int(np.sum(leaf_cols < j))
        assert cx[0, j] == lc
        assert cx[1, j] == lo[lc - ni]
        assert cx[2, j] == int(np.sum(tree_cols < j))
    assert cx[1, m] == n_lo
    cnt = [int(cx[1, j + 1] - cx[1, j] + cx[2, j + 1] - cx[2, j]) for j in range(m)]
    want = sorted(range(m), key=lambda j: (-cnt[j], j))
    assert cx[3, :m].tolist() == want
    # leaf positions of column j are contiguous, and so its leaf occurrences
    pos = {c: p for p, c in enumerate(at)}
    for j in range(m):
        ps = [pos[c] for c in range(ni, n1) if v["col"][c] == j]
        assert ps == list(range(int(cx[0, j]), int(cx[0, j + 1])))
        assert sum(len(occ[p]) for p in ps) == cnt[j] - int(cx[2, j + 1] - cx[2, j])
    # children ranges: tree code h's children are tchild[h] .. tchild[h+1]-1
    hrow = lambda c: c if c < ni else c - n1 + ni
    tch = v["tchild"]
    assert len(tch) == len(tree) + 1
    for h, c in enumerate(tree):
        kids = [x for x in range(n1, nc) if v["parent"][x] == c]
        assert kids == list(range(int(tch[hrow(c)]), int(tch[hrow(c) + 1])))


def walk_decode(v):
    rows = []
    span, dc = v["span"], v["dc"]
    bits = v["val"].view(np.uint32)
    for r in range(len(span) - 1):
        row = []
        for c in dc[span[r]:span[r + 1]]:
            seq = []
            x = int(c)
            while x != 0xFFFFFFFF:
                seq.append((int(v["col"][x]), int(bits[x])))
                x = int(v["parent"][x])
            row.extend(seq[::-1])
        rows.append(row)
    return rows


BATCHES = [
    ("tiny", dict(n_rows=12, n_cols=9, density=0.9, n_values=2, prefix_copy=0.8)),
    ("tiny", dict(n_rows=30, n_cols=20, density=0.5, n_values=3, prefix_copy=0.5)),
    ("tiny", dict(n_rows=3, n_cols=4, density=0.0, n_values=1)),
    ("tiny", dict(n_rows=1, n_cols=50, density=1.0, n_values=1)),
]


def _tiny_csrs():
    out = []
    for i, (_, spec) in enumerate(BATCHES):
        rp, c, v = tiny_batch(77 + i, zeros=True, **{**spec, "n_cols": 50})
        out.append((spec["n_rows"], rp, c, v))
    return out


@pytest.mark.parametrize("flags", [0, T.TOC_UPLOAD_KEEP_DEAD])
def test_image_invariants_and_walk(flags):
    csrs = _tiny_csrs()
    B = config_batches("c1", 0, 1)
    csrs.append(B.batch(0)[:1] + B.batch(0)[1:])
    n_cols = 68
    csrs = [(n, rp, c, v) for (n, rp, c, v) in csrs]
    # pad tiny batches to the same n_cols as c1
    encs, oracle_rows = [], []
    for n, rp, c, v in csrs:
        encs.append(T.toc_encode(n, n_cols, rp, c, v))
        oracle_rows.append(O.canonicalize(n, n_cols, rp, c, v))
    size = T.toc_upload_size(encs, flags)
    buf = np.zeros(size, np.uint8)
    dev = T.toc_upload(encs, buf, flags | T.TOC_UPLOAD_HOST)
    img = read_image(dev, buf)
    assert img["info"]["n_batches"] == len(encs)
    nnz_base = 0
    for b, rows in enumerate(oracle_rows):
        v = batch_view(img, b)
        check_invariants(v)
        assert walk_decode(v) == rows
        assert int(v["t"]["nnz_base"]) == nnz_base
        nnz_base += sum(len(r) for r in rows)
        I, D, N = O.encode(rows)
        st = O.layout_stats(I, D)
        if flags & T.TOC_UPLOAD_KEEP_DEAD:
            assert int(v["t"]["n_codes"]) == N - 1
        else:
            assert int(v["t"]["n_codes"]) == st["n_live"]
            assert int(v["t"]["n_levels"]) == st["max_depth"]
    assert img["info"]["nnz"] == nnz_base


def test_image_products_match_oracle():
    """fp64 products computed by walking the image equal the oracle's."""
    B = config_batches("c1", 0, 1)
    n, rp, cc, vv = B.batch(0)
    enc = T.toc_encode(n, B.n_cols, rp, cc, vv)
    buf = np.zeros(T.toc_upload_size([enc]), np.uint8)
    dev = T.toc_upload([enc], buf, T.TOC_UPLOAD_HOST)
    im = batch_view(read_image(dev, buf), 0)
    rng = np.random.default_rng(0)
    W = rng.standard_normal((B.n_cols, 2))
    G = rng.standard_normal((n, 2))
    nc = len(im["col"])
    H = np.zeros((nc, 2))
    for c in range(nc):
        p = int(im["parent"][c])
        H[c] = im["val"][c] * W[im["col"][c]] + (H[p] if p != 0xFFFFFFFF else 0)
    R = np.array([H[im["dc"][im["span"][r]:im["span"][r + 1]]].sum(0) for r in range(n)])
    rows = O.canonicalize(n, B.n_cols, rp, cc, vv)
    R_o, S = O.dense_right(rows, B.n_cols, W)
    assert np.all(np.abs(R - R_o) <= 1e-12 * S)
    H = np.zeros((nc, 2))
    for r in range(n):
        for x in im["dc"][im["span"][r]:im["span"][r + 1]]:
            H[x] += G[r]
    out = np.zeros((B.n_cols, 2))
    for c in range(nc - 1, -1, -1):
        out[im["col"][c]] += im["val"][c] * H[c]
        p = int(im["parent"][c])
        if p != 0xFFFFFFFF:
            H[p] += H[c]
    out_o, S = O.dense_left(rows, B.n_cols, G)
    assert np.all(np.abs(out - out_o) <= 1e-12 * S)


def test_upload_errors():
    e1 = T.toc_encode(1, 3, [0, 1], [0], np.ones(1, np.float32))
    e2 = T.toc_encode(1, 4, [0, 1], [0], np.ones(1, np.float32))
    with pytest.raises(T.TocError) as ei:
        T.toc_upload_size([e1, e2])
    assert ei.value.status == T.TOC_EINVAL
    size = T.toc_upload_size([e1])
    with pytest.raises(T.TocError) as ei:
        T.toc_upload([e1], np.zeros(size - 1, np.uint8), T.TOC_UPLOAD_HOST)
    assert ei.value.status == T.TOC_ESIZE
    with pytest.raises(T.TocError) as ei:
        T.toc_upload_size([e1], 1 << 7)
    assert ei.value.status == T.TOC_EINVAL


def test_host_image_rejected_by_device_ops():
    e1 = T.toc_encode(1, 3, [0, 1], [0], np.ones(1, np.float32))
    buf = np.zeros(T.toc_upload_size([e1]), np.uint8)
    dev = T.toc_upload([e1], buf, T.TOC_UPLOAD_HOST)
    lib = T.lib()
    assert lib.toc_right_mul(dev.handle, 8, 1, 1, 8, 1, None, 0, None) == T.TOC_EINVAL
    assert "host" in lib.toc_last_error().decode()
    assert lib.toc_decode_csr(dev.handle, 8, 8, 8, None) == T.TOC_EINVAL
    assert lib.toc_map_values(dev.handle, 0, 2.0, None) == T.TOC_EINVAL
    assert lib.toc_decode_dense(dev.handle, 0.0, 8, 3, None) == T.TOC_EINVAL


def test_mlp_host_checks():
    """The neural-network step's checks that need no GPU: an image in host memory
    is rejected; the workspace size is 4 (max rows) (2 h1 + 2 h2 + n_out) bytes
    when the table rows fit in LDS."""
    import ctypes as C
    B = config_batches("c5", 0, 2)
    encs = T.toc_encode_batches(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    hbuf = np.zeros(T.toc_upload_size(encs, T.TOC_UPLOAD_HOST), np.uint8)
    hdev = T.toc_upload(encs, hbuf, T.TOC_UPLOAD_HOST)
    assert T.toc_mlp_workspace_size(hdev, 200, 50, 10) == 4 * 250 * (400 + 100 + 10)
    dummy = C.c_void_p(16)
    st = T.lib().toc_mlp_epoch(hdev.handle, 0, 2, 8, 3, 2, dummy, dummy, dummy, dummy, dummy,
                               dummy, dummy, C.c_float(0.1), dummy, 1 << 20, None)
    assert st == T.TOC_EINVAL
