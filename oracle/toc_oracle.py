"""Plain, slow, obviously correct TOC oracle (TEST INFRASTRUCTURE ONLY).

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may use this
module.  It shares no code with the HIP path and imports nothing from it.

Paper: Li et al., "Tuple-oriented Compression for Large-scale Mini-batch Stochastic
Gradient Descent", arXiv 1702.06943.

Representation used throughout: a mini-batch is a list of rows; a row is a list of
column_index:value pairs ``(col, bits)`` in increasing column order, where ``bits``
is the IEEE-754 binary32 bit pattern of the value (keys compare on bits).
Columns are 0-based (the paper's worked example is 1-based).
"""

from __future__ import annotations

import math
import struct

import numpy as np
import scipy.sparse


class TocInputError(ValueError):
    """Raised for inputs the sparse encoding cannot represent."""


def f32_bits(x: float) -> int:
    """Bit pattern of x rounded to binary32."""
    return struct.unpack("<I", struct.pack("<f", x))[0]


def bits_f32(b: int) -> float:
    """Value (as a Python float, exact) of a binary32 bit pattern."""
    return struct.unpack("<f", struct.pack("<I", b))[0]


# ---------------------------------------------------------------------------
# Sparse encoding (§3, first paragraphs): drop zeros, prefix each nonzero with its
# column index.  Our readings: values are binary32, a value compares equal to zero
# (+0.0 or -0.0) is dropped, NaN/Inf are rejected, columns must be strictly
# increasing inside a row (the pairs come from scanning a dense row left to right).
# ---------------------------------------------------------------------------
def canonicalize(n_rows, n_cols, rowptr, col, val):
    """CSR (rowptr, col, val as float32) -> list of rows of (col, bits) pairs."""
    rowptr = np.asarray(rowptr, dtype=np.int64)
    col = np.asarray(col, dtype=np.int64)
    val = np.asarray(val, dtype=np.float32)
    if n_rows < 0 or n_cols < 0:
        raise TocInputError("negative shape")
    if rowptr.shape != (n_rows + 1,):
        raise TocInputError("rowptr must have n_rows + 1 entries")
    if rowptr[0] != 0 or np.any(np.diff(rowptr) < 0):
        raise TocInputError("rowptr must start at 0 and be non-decreasing")
    nnz = int(rowptr[-1])
    if col.shape != (nnz,) or val.shape != (nnz,):
        raise TocInputError("col/val length must equal rowptr[n_rows]")
    rows = []
    for i in range(n_rows):
        row = []
        prev = -1
        for p in range(int(rowptr[i]), int(rowptr[i + 1])):
            c = int(col[p])
            v = float(val[p])
            if c < 0 or c >= n_cols:
                raise TocInputError("column index out of range")
            if c <= prev:
                raise TocInputError("columns must be strictly increasing in a row")
            prev = c
            if math.isnan(v) or math.isinf(v):
                raise TocInputError("non-finite value")
            if v == 0.0:
                continue
            row.append((c, f32_bits(v)))
        rows.append(row)
    return rows


# ---------------------------------------------------------------------------
# Logical encoding (§3.1, Algorithm 1), written from its two rules:
#  * the tree C starts with every distinct pair of the batch as a child of the
#    root, numbered 1, 2, ... in order of first appearance;
#  * each tuple is cut greedily into the longest sequences C already holds
#    (read from the root down); the code of a piece is the node it ends at, and
#    after every piece that does not end the tuple, C learns that piece followed
#    by the tuple's next pair as a new node (the next number in turn).
# C is one dict (node, pair) -> child: §3.1.1's per-node child map with the node
# folded into the key.
# ---------------------------------------------------------------------------
def _deepest_prefix(children, t, start):
    """The node of the longest sequence of C that t[start:] begins with, and the
    position just past it.  Every pair is a child of the root, so the sequence
    has at least one pair."""
    node, end = 0, start
    while end < len(t) and (node, t[end]) in children:
        node = children[(node, t[end])]
        end += 1
    return node, end


def encode(rows):
    """§3.1 encoding.  rows -> (I, D, N).

    I: list of (col, bits), the first layer of C in node-index order (nodes 1..|I|).
    D: list (one per row) of lists of node indices.
    N: number of nodes of C including the root (= next sequence number).
    """
    children = {}
    I = []
    for t in rows:
        for pair in t:
            if (0, pair) not in children:
                I.append(pair)
                children[(0, pair)] = len(I)
    n_nodes = len(I) + 1
    D = []
    for t in rows:
        codes, start = [], 0
        while start < len(t):
            node, start = _deepest_prefix(children, t, start)
            codes.append(node)
            if start < len(t):            # the piece plus the next pair becomes a node
                children[(node, t[start])] = n_nodes
                n_nodes += 1
        D.append(codes)
    return I, D, n_nodes


# ---------------------------------------------------------------------------
# Decoding tree C' (§4.1.2, Algorithm 2, Table 4), from the same node-creation
# rule: node 1..|I| is the root's child with pair I[i-1]; each later node was made
# when a tuple's code p was followed by a code q, as p's sequence extended by the
# first pair of q's sequence, so it is p's child with that pair as its key.  Nodes
# are numbered in creation order, which D replays tuple by tuple, code by code.
# depth is the length of a node's sequence.
# ---------------------------------------------------------------------------
def build_cprime(I, D):
    """Returns dict with lists parent, key (pairs), depth; index 0 = root."""
    parent, key, depth = [None], [None], [0]
    first = [None]                        # first pair of each node's sequence
    for pair in I:
        parent.append(0)
        key.append(pair)
        depth.append(1)
        first.append(pair)
    for codes in D:
        for p, q in zip(codes[:-1], codes[1:]):
            parent.append(p)
            depth.append(depth[p] + 1)
            first.append(first[p])
            # q may be the node made right here (a tuple repeating its pair): its
            # first pair is then p's, appended just above
            key.append(first[q])
    return {"parent": parent, "key": key, "depth": depth, "n_nodes": len(parent)}


# ---------------------------------------------------------------------------
# Full decode (§4.5, Algorithm 6 without its densify-and-add-c step): a code
# stands for the pairs on the path from the root of C' down to it; a tuple is
# its codes' sequences one after another.  A parent is made before its children,
# so the sequences fill in index order.
# ---------------------------------------------------------------------------
def decode(I, D):
    """(I, D) -> rows of (col, bits) pairs."""
    cp = build_cprime(I, D)
    parent, key = cp["parent"], cp["key"]
    seq = [()] * cp["n_nodes"]
    for node in range(1, cp["n_nodes"]):
        seq[node] = seq[parent[node]] + (key[node],)
    return [[pair for code in d for pair in seq[code]] for d in D]


def decoded_to_csr(rows):
    """rows of (col, bits) -> (rowptr int64, col int32, val float32) arrays."""
    rowptr = np.zeros(len(rows) + 1, dtype=np.int64)
    cols, bits = [], []
    for i, r in enumerate(rows):
        rowptr[i + 1] = rowptr[i] + len(r)
        for c, b in r:
            cols.append(c)
            bits.append(b)
    col = np.asarray(cols, dtype=np.int32)
    val = np.asarray(bits, dtype=np.uint32).view(np.float32)
    return rowptr, col, val


def _coo(rows):
    """rows -> (row index, col, value fp64) arrays of the nonzeros."""
    ri, ci, vi = [], [], []
    for i, r in enumerate(rows):
        for c, b in r:
            ri.append(i)
            ci.append(c)
            vi.append(bits_f32(b))
    return (np.asarray(ri, dtype=np.int64), np.asarray(ci, dtype=np.int64),
            np.asarray(vi, dtype=np.float64))


# ---------------------------------------------------------------------------
# Sparse-safe element-wise operations (§4.2, Algorithm 3): every distinct
# (column, value) pair of A is an entry of I, so A.*c (and A.^2, "similar" by the
# same section) is computed by scanning I and changing each value.  Values are
# binary32, so the new value is the binary32 rounding of the product; a product
# that rounds to zero stays an entry (the structure of A is not revisited).
# ---------------------------------------------------------------------------
MAP_SCALE = 0
MAP_SQUARE = 1


def map_values(I, op, c=1.0):
    """Algorithm 3: I -> I' with every value v replaced by v*c (MAP_SCALE) or v*v
    (MAP_SQUARE), rounded to binary32."""
    out = []
    for col, b in I:
        v = np.float32(bits_f32(b))
        if op == MAP_SCALE:
            w = np.float32(v * np.float32(c))
        elif op == MAP_SQUARE:
            w = np.float32(v * v)
        else:
            raise ValueError("unknown op")
        out.append((col, int(np.asarray(w, dtype=np.float32).view(np.uint32))))
    return out


# ---------------------------------------------------------------------------
# Sparse-unsafe element-wise plus (§4.5, Algorithm 9): decode A fully (decode
# above), densify it, and add c to every element, the
# zeros included.  In binary32: R[i, j] = a_ij + c rounded to binary32.
# ---------------------------------------------------------------------------
def dense_plus(rows, n_cols, c=0.0):
    """Decoded rows -> dense (n_rows, n_cols) float32 array A .+ c."""
    A = np.zeros((len(rows), n_cols), dtype=np.float32)
    for i, r in enumerate(rows):
        for col, b in r:
            A[i, col] = np.float32(bits_f32(b))
    return (A + np.float32(c)).astype(np.float32)


# ---------------------------------------------------------------------------
# Reference products.  Theorems 1 and 2 (and their matrix forms in the appendix)
# state that the TOC algorithms compute exactly A.W and M.A; so the reference is the
# plain definition over the nonzeros of the decoded batch, in fp64:
#   R[i, q]   = sum_j a_ij w_jq         (right multiplication, A.W)
#   out[j, q] = sum_i a_ij g_iq         (left multiplication G^T.A, stored transposed)
# The tolerance scales are the same sums of absolute values of the terms.
# ---------------------------------------------------------------------------
def densify(rows, n_cols):
    """Decoded rows -> the dense fp64 (n_rows, n_cols) matrix A (zeros included),
    on which A.W and A^T.G are plain matmuls."""
    A = np.zeros((len(rows), n_cols))
    for i, r in enumerate(rows):
        for c, b in r:
            A[i, c] = bits_f32(b)
    return A


def _sparse(rows, n_cols):
    """The decoded batch as an fp64 sparse matrix A (n_rows x n_cols)."""
    ri, ci, vi = _coo(rows)
    return scipy.sparse.csr_matrix((vi, (ri, ci)), shape=(len(rows), n_cols))


def dense_right(rows, n_cols, W):
    """R = A.W and S_R = |A|.|W| in fp64 (a sparse-times-dense matmul of the
    decoded batch).  W: (n_cols, k)."""
    W = np.asarray(W, dtype=np.float64)
    if W.ndim != 2 or W.shape[0] != n_cols:
        raise TocInputError("W must be n_cols x k")
    A = _sparse(rows, n_cols)
    R = np.asarray(A @ W, dtype=np.float64).reshape(len(rows), W.shape[1])
    S = np.asarray(abs(A) @ np.abs(W), dtype=np.float64).reshape(len(rows), W.shape[1])
    return R, S


def dense_left(rows, n_cols, G):
    """out = (G^T.A)^T = A^T.G (n_cols x k) and S_out = |A|^T.|G| in fp64 (a
    sparse-times-dense matmul of the decoded batch).  G: (n_rows, k)."""
    G = np.asarray(G, dtype=np.float64)
    if G.ndim != 2 or G.shape[0] != len(rows):
        raise TocInputError("G must be n_rows x k")
    At = _sparse(rows, n_cols).T.tocsr()
    out = np.asarray(At @ G, dtype=np.float64).reshape(n_cols, G.shape[1])
    S = np.asarray(abs(At) @ np.abs(G), dtype=np.float64).reshape(n_cols, G.shape[1])
    return out, S


# ---------------------------------------------------------------------------
# The products through C' (Theorems 1 and 2, the content of Algorithms 4, 5, 7
# and 8), in fp64, used to check those theorems against the plain products above.
# Both rest on two objects:
#  * H[n]: node n's sequence applied to W, i.e. the sum of val * W[col] over the
#    pairs on the path from the root to n; a parent is made before its children,
#    so H fills in index order from H[parent];
#  * M: the tuple-by-node count matrix of D (M[i, n] = how often tuple i uses n).
# Right (Theorem 1): A W = M H.  Left (Theorem 2): a pair of node n's sequence is
# used by every tuple that uses n or one of n's descendants, so column col(n) of
# A^T G gains val(n) times the sum of (M^T G) over n and its descendants.
# ---------------------------------------------------------------------------
def _occurrences(D, n_nodes):
    """M as a scipy sparse matrix (duplicates summed)."""
    rows = [i for i, d in enumerate(D) for _ in d]
    codes = [c for d in D for c in d]
    return scipy.sparse.csr_matrix((np.ones(len(codes)), (rows, codes)), shape=(len(D), n_nodes))


def toc_right(I, D, W):
    """Theorem 1: R = M H."""
    W = np.asarray(W, dtype=np.float64)
    cp = build_cprime(I, D)
    parent, key = cp["parent"], cp["key"]
    H = np.zeros((cp["n_nodes"], W.shape[1]))
    for n in range(1, cp["n_nodes"]):
        col, bits = key[n]
        H[n] = H[parent[n]] + bits_f32(bits) * W[col]
    return np.asarray(_occurrences(D, cp["n_nodes"]) @ H)


def toc_left(I, D, G, n_cols):
    """Theorem 2: out[col(n)] += val(n) * (sum of M^T G over n's subtree)."""
    G = np.asarray(G, dtype=np.float64)
    cp = build_cprime(I, D)
    parent, key = cp["parent"], cp["key"]
    sub = np.asarray(_occurrences(D, cp["n_nodes"]).T @ G)
    for n in range(cp["n_nodes"] - 1, 0, -1):   # children before their parents
        sub[parent[n]] += sub[n]
    out = np.zeros((n_cols, G.shape[1]))
    for n in range(1, cp["n_nodes"]):
        col, bits = key[n]
        out[col] += bits_f32(bits) * sub[n]
    return out


# ---------------------------------------------------------------------------
# Sizes.
# ---------------------------------------------------------------------------
def layout_stats(I, D):
    """Counts that define the canonical compressed size of a batch.

    live: codes referenced by D plus all their ancestors (the only codes any of the
    operations of §4 touch); max_depth over live codes; canonical bytes
      B_toc = 4|D| + 4(n+1) + 10 live + 4 (max_depth + 1)
    i.e. a u32 per code occurrence, a u32 per row boundary, (u32 parent, u16 column,
    f32 value) per live code and a u32 per level boundary.
    """
    cp = build_cprime(I, D)
    parent, depth = cp["parent"], cp["depth"]
    live = [False] * cp["n_nodes"]
    stack = [c for d in D for c in d]
    while stack:
        c = stack.pop()
        if c != 0 and not live[c]:
            live[c] = True
            stack.append(parent[c])
    n_live = sum(live)
    max_depth = max((depth[c] for c in range(cp["n_nodes"]) if live[c]), default=0)
    n_codes = sum(len(d) for d in D)
    n_deep = sum(1 for c in range(cp["n_nodes"]) if live[c] and depth[c] >= 2)
    canon = 4 * n_codes + 4 * (len(D) + 1) + 10 * n_live + 4 * (max_depth + 1)
    return {
        "n_rows": len(D),
        "n_first": len(I),
        "n_codes": n_codes,
        "n_nodes": cp["n_nodes"],
        "n_live": n_live,
        "n_deep": n_deep,
        "max_depth": max_depth,
        "canon_bytes": canon,
    }


def level_order(I, D):
    """The live codes in level order, as the operations of §4 can read them.

    Live codes are those D references plus all their ancestors (the only codes
    Algorithms 4-8 touch).  Sorted stably by (depth, index), every parent comes
    before its children, which is all the forward scan of Algorithm 4 and the
    backward scan of Algorithm 5 need.  Returns a dict: per live code in that order
    parent (new index, None at depth 1), key (col, bits), depth; level_off[d] =
    number of live codes of depth <= d (d = 0..max depth); D renumbered.
    """
    cp = build_cprime(I, D)
    parent, depth = cp["parent"], cp["depth"]
    live = set()
    for d in D:
        for c in d:
            while c != 0 and c not in live:
                live.add(c)
                c = parent[c]
    order = sorted(live, key=lambda c: (depth[c], c))
    new = {c: i for i, c in enumerate(order)}
    max_depth = max((depth[c] for c in order), default=0)
    level_off = [sum(1 for c in order if depth[c] <= d) for d in range(max_depth + 1)]
    return {
        "parent": [new[parent[c]] if depth[c] > 1 else None for c in order],
        "key": [cp["key"][c] for c in order],
        "depth": [depth[c] for c in order],
        "level_off": level_off,
        "D": [[new[c] for c in d] for d in D],
        "order": order,
    }


def _packed_array_bytes(values):
    """Bit packing of §3.2: ceil(log2(max+1)/8) bytes per integer (at least one),
    plus a header holding the count (u32) and the bytes per integer (u8)."""
    mx = max(values, default=0)
    width = max(1, math.ceil(math.log2(mx + 1) / 8)) if mx > 0 else 1
    return 5 + width * len(values)


def physical_bytes(I, D):
    """Physical encoding of §3.2: I's columns bit-packed, I's values replaced by
    indices into an array of unique values (4 bytes each) which are bit-packed,
    D's codes concatenated and bit-packed, tuple start offsets bit-packed."""
    uniq = sorted(set(b for _, b in I))
    where = {b: q for q, b in enumerate(uniq)}
    size = _packed_array_bytes([c for c, _ in I])
    size += 5 + 4 * len(uniq)
    size += _packed_array_bytes([where[b] for _, b in I])
    size += _packed_array_bytes([c for d in D for c in d])
    starts = [0]
    for d in D:
        starts.append(starts[-1] + len(d))
    size += _packed_array_bytes(starts)
    return size


# ---------------------------------------------------------------------------
# Sizes of the TOC variants compared in the ablation study of §5.2 (compression
# ratios of TOC_SPARSE, TOC_SPARSE_AND_LOGICAL and TOC_FULL against the dense
# encoding DEN).  The paper names the variants but not their byte layouts; the
# reading taken here: DEN stores n x m binary32 values; the sparse encoding (§3)
# stores each nonzero as a u32 column index and a binary32 value, plus n + 1 u32
# tuple starts; the logical encoding (§3.1) stores I as such pairs, D's codes as
# u32 and n + 1 u32 tuple starts; TOC_FULL is the physical encoding of §3.2.
# ---------------------------------------------------------------------------
def dense_bytes(n_rows, n_cols):
    return 4 * n_rows * n_cols


def sparse_bytes(rows):
    return 8 * sum(len(t) for t in rows) + 4 * (len(rows) + 1)


def logical_bytes(I, D):
    return 8 * len(I) + 4 * sum(len(d) for d in D) + 4 * (len(D) + 1)


# ---------------------------------------------------------------------------
# Physical encoding as bytes, §3.2.  The paper fixes the techniques -- bit packing
# with ceil(log2(max+1)/8) bytes per integer behind a header that gives the count
# and the bytes per integer, value indexing of I's values, D's codes of all tuples
# concatenated, and the tuple starting indexes -- but not the byte layout.  The
# reading taken here: five arrays in the order I's columns, the unique values,
# I's value indexes, D's codes, the tuple starts (n_rows + 1 offsets into D, the
# last one |D|); each behind a 5-byte header (count as a little-endian u32, then
# the bytes per integer as a u8); integers little-endian in that many bytes; the
# unique values are the distinct binary32 bit patterns of I's values in
# ascending order, 4 bytes each.  §4.1.1 reads such integers back by copying
# their bytes into a wider integer.
# ---------------------------------------------------------------------------
def _width(mx):
    """Bytes per integer for an array whose largest value is mx: ceil(log2(mx+1)/8),
    at least one (bit_length is ceil(log2(mx+1)) exactly)."""
    return max(1, (int(mx).bit_length() + 7) // 8)


def _pack_array(values, width=None):
    w = _width(max(values, default=0)) if width is None else width
    out = bytearray(struct.pack("<IB", len(values), w))
    for v in values:
        out += int(v).to_bytes(w, "little")
    return bytes(out)


def _unpack_array(blob, pos):
    if pos + 5 > len(blob):
        raise TocInputError("truncated array header")
    n, w = struct.unpack_from("<IB", blob, pos)
    pos += 5
    if not 1 <= w <= 4:
        raise TocInputError("bytes per integer must be 1..4")
    if pos + n * w > len(blob):
        raise TocInputError("truncated array")
    vals = [int.from_bytes(blob[pos + q * w:pos + (q + 1) * w], "little") for q in range(n)]
    return vals, pos + n * w


def pack_physical(I, D):
    """(I, D) -> bytes of the physical encoding (reading above)."""
    uniq = sorted(set(b for _, b in I))
    where = {b: q for q, b in enumerate(uniq)}
    starts = [0]
    for d in D:
        starts.append(starts[-1] + len(d))
    blob = _pack_array([c for c, _ in I])
    blob += _pack_array(uniq, width=4)
    blob += _pack_array([where[b] for _, b in I])
    blob += _pack_array([c for d in D for c in d])
    blob += _pack_array(starts)
    return blob


def unpack_physical(blob):
    """Bytes of the physical encoding -> (I, D); raises TocInputError on a
    malformed input."""
    cols, p = _unpack_array(blob, 0)
    if p + 5 <= len(blob) and blob[p + 4] != 4:
        raise TocInputError("unique values are 4 bytes each")
    uniq, p = _unpack_array(blob, p)
    vidx, p = _unpack_array(blob, p)
    codes, p = _unpack_array(blob, p)
    starts, p = _unpack_array(blob, p)
    if p != len(blob):
        raise TocInputError("trailing bytes")
    if len(vidx) != len(cols) or any(q >= len(uniq) for q in vidx):
        raise TocInputError("bad value indexes")
    if not starts or starts[0] != 0 or starts[-1] != len(codes) or \
            any(b < a for a, b in zip(starts, starts[1:])):
        raise TocInputError("bad tuple starts")
    I = [(c, uniq[q]) for c, q in zip(cols, vidx)]
    D = [codes[starts[r]:starts[r + 1]] for r in range(len(starts) - 1)]
    return I, D


# ---------------------------------------------------------------------------
# Mini-batch gradient descent on a TOC batch, §2.1: one step moves the model h by
# the learning rate times the mean, over the batch's tuples, of the loss gradient
# (the MGD update equation).  For the linear models of Table 1 the loss of a tuple
# (x, y) depends on h through r = x^T h only, so the batch gradient is
# A^T g / |B| with g_i = d loss / d r at r_i = (A h)_i: the paper's linear
# regression example, ((A h - Y)^T A)^T, is the case g = r - y.  Losses (Table 1's
# caption names them; the label convention is a reading): squared 1/2 (y - r)^2;
# logistic log(1 + exp(-y r)) with y in {-1, +1}; hinge max(0, 1 - y r) with
# y in {-1, +1}, whose subgradient at y r = 1 is taken as 0.
# ---------------------------------------------------------------------------
MGD_LINEAR, MGD_LOGISTIC, MGD_HINGE = 0, 1, 2


def mgd_loss(loss, r, y):
    """Per-tuple loss values (fp64 arrays)."""
    r, y = np.asarray(r, np.float64), np.asarray(y, np.float64)
    if loss == MGD_LINEAR:
        return 0.5 * (y - r) ** 2
    if loss == MGD_LOGISTIC:
        return np.logaddexp(0.0, -y * r)            # log(1 + exp(-y r)) without overflow
    if loss == MGD_HINGE:
        return np.maximum(0.0, 1.0 - y * r)
    raise TocInputError("unknown loss")


def mgd_dloss(loss, r, y):
    """d loss / d r per tuple (fp64 arrays)."""
    r, y = np.asarray(r, np.float64), np.asarray(y, np.float64)
    if loss == MGD_LINEAR:
        return r - y
    if loss == MGD_LOGISTIC:
        # -y / (1 + exp(y r)) = -y * sigmoid(-y r), the sigmoid as (1 + tanh(z/2)) / 2
        return -y * 0.5 * (1.0 + np.tanh(-0.5 * y * r))
    if loss == MGD_HINGE:
        return np.where(y * r < 1.0, -y, 0.0)
    raise TocInputError("unknown loss")


def mgd_step(rows, n_cols, h, y, loss, lr):
    """One MGD step on a decoded batch: returns the new model (fp64) and the
    tolerance scale |A|^T (|g| + |A||h|) of each component (sums of absolute
    terms).  A batch without tuples leaves h unchanged."""
    h = np.asarray(h, np.float64)
    if len(rows) == 0:
        return h.copy(), np.zeros_like(h)
    r, s_r = dense_right(rows, n_cols, h[:, None])
    g = mgd_dloss(loss, r[:, 0], y)
    grad, _ = dense_left(rows, n_cols, g[:, None])
    _, scale = dense_left(rows, n_cols, (np.abs(g) + s_r[:, 0])[:, None])
    return h - lr / len(rows) * grad[:, 0], scale[:, 0]


# ---------------------------------------------------------------------------
# Mini-batch gradient descent for the neural network of §5.1 (the NN row of
# Table 1, whose matrix operations are A.M and M.A): a feed-forward network with
# two hidden layers (sigmoid activations) and a sigmoid output for one class or
# a softmax output for several, trained with cross-entropy loss.  The batch's
# first layer is Z1 = A W1 + b1 (A.M with M = W1) and its weight gradient is
# A^T dZ1 (M.A with M = dZ1^T).  Readings: every layer has a bias; the loss is the
# mean over the batch's tuples, so one step moves every parameter by lr times the
# gradient of that mean (§2.1's update); labels are class indexes (0/1 for the
# single sigmoid output).
# ---------------------------------------------------------------------------
def _sigmoid(x):
    return 0.5 * (1.0 + np.tanh(0.5 * x))


def _mlp_forward(A, p):
    H1 = _sigmoid(A @ p["W1"] + p["b1"])
    H2 = _sigmoid(H1 @ p["W2"] + p["b2"])
    Z3 = H2 @ p["W3"] + p["b3"]
    return H1, H2, Z3


def mlp_loss(rows, n_cols, params, labels):
    """Mean cross-entropy loss of the network on a decoded batch (fp64)."""
    p = {k: np.asarray(v, np.float64) for k, v in params.items()}
    labels = np.asarray(labels, np.int64)
    _, _, Z3 = _mlp_forward(densify(rows, n_cols), p)
    if Z3.shape[1] == 1:
        z = Z3[:, 0]
        per = np.logaddexp(0.0, z) - labels * z        # -log sigmoid(z) or -log(1 - sigmoid(z))
    else:
        zmax = Z3.max(axis=1, keepdims=True)
        lse = zmax[:, 0] + np.log(np.exp(Z3 - zmax).sum(axis=1))
        per = lse - Z3[np.arange(len(labels)), labels]
    return float(per.mean()) if len(per) else 0.0


def mlp_step(rows, n_cols, params, labels, lr):
    """One MGD step of the network on a decoded batch: returns (new parameters,
    gradients of the mean loss), both dicts of fp64 arrays keyed W1, b1, W2, b2, W3,
    b3.  A batch without tuples leaves the parameters unchanged."""
    p = {k: np.asarray(v, np.float64) for k, v in params.items()}
    n = len(rows)
    if n == 0:
        return {k: v.copy() for k, v in p.items()}, {k: np.zeros_like(v) for k, v in p.items()}
    labels = np.asarray(labels, np.int64)
    A = densify(rows, n_cols)
    H1, H2, Z3 = _mlp_forward(A, p)
    C = Z3.shape[1]
    if C == 1:
        P = _sigmoid(Z3)
        Y = labels[:, None].astype(np.float64)
    else:
        E = np.exp(Z3 - Z3.max(axis=1, keepdims=True))
        P = E / E.sum(axis=1, keepdims=True)
        Y = np.zeros_like(P)
        Y[np.arange(n), labels] = 1.0
    dZ3 = (P - Y) / n                                   # d (mean loss) / d Z3
    dZ2 = (dZ3 @ p["W3"].T) * H2 * (1.0 - H2)
    dZ1 = (dZ2 @ p["W2"].T) * H1 * (1.0 - H1)
    g = {"W3": H2.T @ dZ3, "b3": dZ3.sum(axis=0),
         "W2": H1.T @ dZ2, "b2": dZ2.sum(axis=0),
         "W1": A.T @ dZ1, "b1": dZ1.sum(axis=0)}
    return {k: p[k] - lr * g[k] for k in p}, g


def mlp_grad_scale(rows, n_cols, params, labels):
    """Scale S of each gradient entry of mlp_step, for the tolerance eps * S of a
    binary32 gradient (like the products' 1e-5 * sum |a_ij w_jq|).  S is the
    backward pass with every factor replaced by its magnitude (|P - Y| for the
    output error, |W| for the weights), each factor weighted by its sensitivity to
    the forward pass's rounding: c_l, the sum of the absolute values of the terms
    of the pre-activations Z_l (with the previous layer's c carried through the
    sigmoid's slope, at most 1/4), bounds the absolute error of Z_l in units of
    eps; an activation H then carries error c/4, the slope H (1 - H) and the
    softmax output relative error of order c.  So every term of every gradient
    entry counts |term| (1 + its factors' c).  Returns a dict keyed like the
    gradients."""
    p = {k: np.asarray(v, np.float64) for k, v in params.items()}
    n = len(rows)
    if n == 0:
        return {k: np.zeros_like(v) for k, v in p.items()}
    labels = np.asarray(labels, np.int64)
    A = densify(rows, n_cols)
    H1, H2, Z3 = _mlp_forward(A, p)
    aW1, aW2, aW3 = np.abs(p["W1"]), np.abs(p["W2"]), np.abs(p["W3"])
    # forward sensitivities (absolute error bounds of Z_l, in units of eps)
    c1 = np.abs(A) @ aW1 + np.abs(p["b1"])
    c2 = H1 @ aW2 + np.abs(p["b2"]) + 0.25 * (c1 @ aW2)
    c3 = H2 @ aW3 + np.abs(p["b3"]) + 0.25 * (c2 @ aW3)
    if Z3.shape[1] == 1:
        P = _sigmoid(Z3)
        Y = labels[:, None].astype(np.float64)
    else:
        E = np.exp(Z3 - Z3.max(axis=1, keepdims=True))
        P = E / E.sum(axis=1, keepdims=True)
        Y = np.zeros_like(P)
        Y[np.arange(n), labels] = 1.0
    # the output error and its sensitivity (a softmax moves by at most 2 P max|dZ|)
    M3 = (np.abs(P - Y) + 2.0 * P * c3.max(axis=1, keepdims=True)) / n
    M2 = (M3 @ aW3.T) * H2 * (1.0 - H2) * (1.0 + c2)
    M1 = (M2 @ aW2.T) * H1 * (1.0 - H1) * (1.0 + c1)
    return {"W3": (H2 + 0.25 * c2).T @ M3, "b3": M3.sum(axis=0),
            "W2": (H1 + 0.25 * c1).T @ M2, "b2": M2.sum(axis=0),
            "W1": np.abs(A).T @ M1, "b1": M1.sum(axis=0)}
