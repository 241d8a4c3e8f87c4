"""Seeded generators for the five synthetic workloads and for small test batches.

Every draw comes from ``np.random.SeedSequence([SEED, config, stream, batch])`` with
stream 0 = A, 1 = W, 2 = G, 3 = per-dataset constants, so any batch can be
regenerated on its own (and in parallel) without drawing the others.

The paper's datasets (Table 5) are not available; these stand in for them:
  c1  250 x 68 dense categorical table (US-Census-like width)
  c2  sparse text, 47,236 columns (Rcv1-like width)
  c3  28 x 28 images, 80 % zeros (Mnist-like)
  c4  dense quantised features, 1,000 columns
  c5  one-hot categorical + numeric fields, 900 columns, 16 M rows (ImageNet-like width)
All batches have 250 rows, the mini-batch size of the paper's experiments.
"""

from __future__ import annotations

import numpy as np

SEED = 170206943

CONFIGS = {
    "c1": dict(cid=1, name="tiny categorical LR batch", n_batches=1, rows=250,
               cols=68, k=1, w_sigma=1.0),
    "c2": dict(cid=2, name="sparse text linear model", n_batches=4000, rows=250,
               cols=47236, k=1, w_sigma=0.01),
    "c3": dict(cid=3, name="image-like MLP first layer", n_batches=40000, rows=250,
               cols=784, k=300, w_sigma=0.05),
    "c4": dict(cid=4, name="dense quantised features, wide hidden layer",
               n_batches=20000, rows=250, cols=1000, k=200, w_sigma=0.05),
    "c5": dict(cid=5, name="one-hot full epoch resident in HBM", n_batches=64000,
               rows=250, cols=900, k=1, w_sigma=1.0),
}


def _rng(cid, stream, batch=0):
    return np.random.default_rng(np.random.SeedSequence([SEED, cid, stream, batch]))


def _zipf_cdf(n_ranks, s):
    p = np.arange(1, n_ranks + 1, dtype=np.float64) ** (-s)
    c = np.cumsum(p)
    return c / c[-1]


def _zipf_draw(rng, cdf, size):
    """0-based ranks of a finite Zipf law by inverse-cdf sampling."""
    r = np.searchsorted(cdf, rng.random(size), side="right")
    return np.minimum(r, len(cdf) - 1)


class Batches:
    """A run of mini-batches in one concatenated CSR.

    rowptr has sum(n_rows)+1 entries and starts at 0; batch b owns rows
    row_off[b]:row_off[b+1].
    """

    def __init__(self, n_cols, n_rows, rowptr, col, val, first_batch=0):
        self.n_cols = int(n_cols)
        self.n_rows = np.asarray(n_rows, dtype=np.int32)
        self.rowptr = np.asarray(rowptr, dtype=np.int64)
        self.col = np.asarray(col, dtype=np.int32)
        self.val = np.asarray(val, dtype=np.float32)
        self.row_off = np.zeros(len(self.n_rows) + 1, dtype=np.int64)
        np.cumsum(self.n_rows, out=self.row_off[1:])
        self.first_batch = first_batch

    @property
    def n_batches(self):
        return len(self.n_rows)

    @property
    def nnz(self):
        return int(self.rowptr[-1])

    def batch(self, b):
        """(n_rows, rowptr starting at 0, col, val) of batch b (views)."""
        r0, r1 = self.row_off[b], self.row_off[b + 1]
        p0, p1 = self.rowptr[r0], self.rowptr[r1]
        return (int(r1 - r0), self.rowptr[r0:r1 + 1] - p0, self.col[p0:p1],
                self.val[p0:p1])

    @staticmethod
    def concat(parts):
        n_cols = parts[0].n_cols
        n_rows = np.concatenate([p.n_rows for p in parts])
        col = np.concatenate([p.col for p in parts])
        val = np.concatenate([p.val for p in parts])
        rowptr = [np.zeros(1, dtype=np.int64)]
        base = 0
        for p in parts:
            rowptr.append(p.rowptr[1:] + base)
            base += p.nnz
        return Batches(n_cols, n_rows, np.concatenate(rowptr), col, val,
                       parts[0].first_batch)


def _dense_to_csr(A):
    """Dense float32 rows -> (rowptr, col, val) keeping entries != 0."""
    mask = A != 0
    counts = mask.sum(axis=1)
    rowptr = np.zeros(A.shape[0] + 1, dtype=np.int64)
    np.cumsum(counts, out=rowptr[1:])
    rr, cc = np.nonzero(mask)
    return rowptr, cc.astype(np.int32), A[rr, cc].astype(np.float32)


def _nonzero_f32(x):
    x = np.asarray(x, dtype=np.float32)
    x[x == 0] = np.float32(0.5)
    return x


# --- c1: tiny categorical table -----------------------------------------------
def _c1_batch(b, rows, cols):
    const = _rng(1, 3)
    vocab = _nonzero_f32(const.uniform(-1.0, 1.0, size=(cols, 8)))
    rng = _rng(1, 0, b)
    cdf = _zipf_cdf(8, 1.2)
    ranks = _zipf_draw(rng, cdf, (rows, cols))
    A = vocab[np.arange(cols)[None, :], ranks]
    copy = rng.random(rows) < 0.6
    for r in range(1, rows):
        src = rng.integers(0, r)
        if copy[r]:
            A[r, :40] = A[src, :40]
    return _dense_to_csr(A)


# --- c2: sparse text ------------------------------------------------------------
_C2_CACHE = {}


def _c2_batch(b, rows, cols):
    if cols not in _C2_CACHE:
        const = _rng(2, 3)
        _C2_CACHE[cols] = (_zipf_cdf(cols, 1.1), const.permutation(cols))
    cdf, perm = _C2_CACHE[cols]
    rng = _rng(2, 0, b)
    nnz = np.minimum(rng.poisson(75.0, size=rows), cols).astype(np.int64)
    n_draw = 3 * nnz + 16
    row_of = np.repeat(np.arange(rows, dtype=np.int64), n_draw)
    cids = perm[_zipf_draw(rng, cdf, int(n_draw.sum()))].astype(np.int64)
    keys = row_of * cols + cids
    uk, first = np.unique(keys, return_index=True)
    order = np.argsort(first, kind="stable")
    kd = uk[order]                               # distinct (row, col) in draw order
    kr = kd // cols
    start = np.searchsorted(kr, np.arange(rows), side="left")
    rank = np.arange(len(kd)) - start[kr]
    kept = np.sort(kd[rank < nnz[kr]])
    r = kept // cols
    c = (kept % cols).astype(np.int32)
    rowptr = np.zeros(rows + 1, dtype=np.int64)
    np.cumsum(np.bincount(r, minlength=rows), out=rowptr[1:])
    q = rng.integers(1, 17, size=len(c))
    return rowptr, c, (q / 16.0).astype(np.float32)


# --- c3: 28x28 blobs --------------------------------------------------------------
_GRID = None


def _c3_batch(b, rows, cols):
    global _GRID
    side = int(round(np.sqrt(cols)))
    assert side * side == cols
    if _GRID is None or _GRID[0].shape[0] != cols:
        yy, xx = np.divmod(np.arange(cols), side)
        _GRID = (xx.astype(np.float64), yy.astype(np.float64))
    xx, yy = _GRID
    keep = int(round(0.2 * cols))
    rng = _rng(3, 0, b)
    centre = rng.normal((side - 1) / 2.0, 2.0, size=(2, rows))
    d2 = (xx[None, :] - centre[0][:, None]) ** 2 + (yy[None, :] - centre[1][:, None]) ** 2
    f = np.exp(-d2 / (2.0 * 4.0 ** 2)) * (1.0 + 0.3 * rng.standard_normal((rows, cols)))
    idx = np.argpartition(-f, keep - 1, axis=1)[:, :keep]
    idx.sort(axis=1)
    fk = np.take_along_axis(f, idx, axis=1)
    lo = fk.min(axis=1, keepdims=True)
    hi = fk.max(axis=1, keepdims=True)
    q = np.clip(np.rint(255.0 * (fk - lo) / np.maximum(hi - lo, 1e-300)), 1, 255)
    rowptr = np.arange(rows + 1, dtype=np.int64) * keep
    return rowptr, idx.ravel().astype(np.int32), q.ravel().astype(np.float32)


# --- c4: dense quantised ------------------------------------------------------------
_C4_CACHE = {}


def _c4_batch(b, rows, cols):
    if cols not in _C4_CACHE:
        const = _rng(4, 3)
        lv = np.sort(np.clip(_nonzero_f32(const.standard_normal((cols, 256))), -9.5, 9.5),
                     axis=1).astype(np.float32)
        flat = (lv.astype(np.float64) + 20.0 * np.arange(cols)[:, None]).ravel()
        _C4_CACHE[cols] = (lv, flat)
    lv, flat = _C4_CACHE[cols]
    rng = _rng(4, 0, b)
    z = np.clip(rng.standard_normal((rows, cols)), -9.5, 9.5)
    shift = 20.0 * np.arange(cols)[None, :]
    pos = np.searchsorted(flat, (z + shift).ravel()).reshape(rows, cols)
    li = np.clip(pos - 256 * np.arange(cols)[None, :], 0, 255)
    A = lv[np.arange(cols)[None, :], li]
    copy = rng.random(rows) < 0.3
    src = rng.integers(0, np.maximum(np.arange(rows), 1))
    pre = min(200, cols)
    for r in range(1, rows):
        if copy[r]:
            A[r, :pre] = A[src[r], :pre]
    return _dense_to_csr(A)


# --- c5: one-hot fields -----------------------------------------------------------
_C5_CACHE = {}


def _c5_fields(cols):
    if cols not in _C5_CACHE:
        const = _rng(5, 3)
        n_num = 10
        n_cat = cols - n_num
        raw = np.rint(np.exp(const.uniform(np.log(2.0), np.log(100.0), size=40)))
        card = np.maximum(2, np.floor(raw * n_cat / raw.sum())).astype(np.int64)
        card[np.argmax(card)] += n_cat - card.sum()
        off = np.zeros(41, dtype=np.int64)
        np.cumsum(card, out=off[1:])
        cdfs = [_zipf_cdf(int(c), 1.2) for c in card]
        _C5_CACHE[cols] = (card, off, cdfs, n_cat)
    return _C5_CACHE[cols]


def _c5_batch(b, rows, cols):
    card, off, cdfs, n_cat = _c5_fields(cols)
    rng = _rng(5, 0, b)
    nf = len(card)
    C = np.empty((rows, nf + 10), dtype=np.int32)
    for f in range(nf):
        C[:, f] = off[f] + _zipf_draw(rng, cdfs[f], rows)
    C[:, nf:] = n_cat + np.arange(10)[None, :]
    V = np.ones((rows, nf + 10), dtype=np.float32)
    V[:, nf:] = rng.integers(1, 65, size=(rows, 10)) / 64.0
    rowptr = np.arange(rows + 1, dtype=np.int64) * (nf + 10)
    return rowptr, C.ravel(), V.ravel()


_MAKERS = {"c1": _c1_batch, "c2": _c2_batch, "c3": _c3_batch, "c4": _c4_batch,
           "c5": _c5_batch}


def config_batches(cfg, first=0, count=None):
    """Mini-batches first..first+count-1 of a workload as one Batches object."""
    spec = CONFIGS[cfg]
    if count is None:
        count = spec["n_batches"] - first
    rows, cols = spec["rows"], spec["cols"]
    parts_rp, parts_c, parts_v, n_rows = [], [], [], []
    base = 0
    for b in range(first, first + count):
        rp, c, v = _MAKERS[cfg](b, rows, cols)
        parts_rp.append(rp[1:] + base if parts_rp else rp + base)
        base += int(rp[-1])
        parts_c.append(c)
        parts_v.append(v)
        n_rows.append(rows)
    if count == 0:
        return Batches(cols, [], np.zeros(1, np.int64), [], [], first)
    return Batches(cols, n_rows, np.concatenate(parts_rp), np.concatenate(parts_c),
                   np.concatenate(parts_v), first)


def dense_normal(shape, sigma, seed_words):
    """fp32 N(0, sigma^2) matrix from a seed sequence."""
    rng = np.random.default_rng(np.random.SeedSequence([SEED] + list(seed_words)))
    return (sigma * rng.standard_normal(shape)).astype(np.float32)


def config_W(cfg, k=None):
    spec = CONFIGS[cfg]
    k = spec["k"] if k is None else k
    return dense_normal((spec["cols"], k), spec["w_sigma"], [spec["cid"], 1])


def config_G(cfg, first=0, count=1, k=None):
    """G rows of batches first..first+count-1 stacked (each batch seeded alone)."""
    spec = CONFIGS[cfg]
    k = spec["k"] if k is None else k
    return np.concatenate(
        [dense_normal((spec["rows"], k), 1.0, [spec["cid"], 2, b])
         for b in range(first, first + count)], axis=0) if count else \
        np.zeros((0, k), np.float32)


def dense_normal_device(shape, sigma, seed, device):
    """fp32 N(0, sigma^2) tensor drawn on a device by torch's seeded generator
    (for operands too large to draw on the host)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    t = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    return t.mul_(sigma)


def tiny_batch(seed, n_rows, n_cols, density=0.5, n_values=3, integer=False,
               zeros=False, prefix_copy=0.0):
    """Small random CSR batch whose values come from a few levels so that pairs
    repeat.  zeros=True plants explicit +0.0 / -0.0 entries (to be dropped);
    prefix_copy makes rows start with a copy of an earlier row's prefix."""
    rng = np.random.default_rng(np.random.SeedSequence([SEED, 99, seed]))
    if integer:
        levels = np.arange(1, n_values + 1, dtype=np.float32) * \
            np.where(rng.random(n_values) < 0.3, -1, 1).astype(np.float32)
    else:
        levels = _nonzero_f32(rng.uniform(-2.0, 2.0, size=n_values))
    A = levels[rng.integers(0, n_values, size=(n_rows, n_cols))]
    A[rng.random((n_rows, n_cols)) >= density] = 0.0
    if prefix_copy > 0 and n_rows > 1:
        for r in range(1, n_rows):
            if rng.random() < prefix_copy:
                src = rng.integers(0, r)
                cut = rng.integers(1, n_cols + 1)
                A[r, :cut] = A[src, :cut]
    if zeros:
        mask = np.zeros_like(A, dtype=bool)
        z = (A == 0) & (rng.random(A.shape) < 0.3)
        mask |= z
        signs = np.where(rng.random(A.shape) < 0.5, np.float32(-0.0), np.float32(0.0))
        rowptr = np.zeros(n_rows + 1, dtype=np.int64)
        cols, vals = [], []
        for r in range(n_rows):
            for c in range(n_cols):
                if A[r, c] != 0:
                    cols.append(c)
                    vals.append(A[r, c])
                elif mask[r, c]:
                    cols.append(c)
                    vals.append(signs[r, c])
            rowptr[r + 1] = len(cols)
        return rowptr, np.asarray(cols, np.int32), np.asarray(vals, np.float32)
    return _dense_to_csr(A)
