"""Plain CPU oracle for tuple-oriented compression (TOC).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call anything in this package.
The product path (``libtoc.so`` and its Python binding) never imports it, and this
package imports nothing from the product.

Everything here follows Li et al., "Tuple-oriented Compression for Large-scale
Mini-batch Stochastic Gradient Descent" (arXiv 1702.06943); each function cites the
section, algorithm, table or equation it restates.  Floating point is fp64.

Parity status of each function (what pins it, see ``tests/test_oracle.py``):
  canonicalize   pinned: sparse-encoding example of §3 (row R2), error cases
  encode         pinned: Table 2 traces + its caption (worked example), brute-force
                 greedy re-encoder on random tiny tables, round trip
  build_cprime   pinned: Table 4 (all 11 nodes), node-count closed form, invariants
  decode         pinned: lossless round trip on random inputs + worked example
  dense_right    pinned: hand-computed worked-example sums, numpy dense matmul on the
                 densified batch, integer exactness
  dense_left     pinned: as dense_right, plus duality <G, A W> = <A^T G, W>
  densify        pinned: equal to a dense matrix filled by the test itself
  toc_right      pinned: Theorem 1 (equals dense_right) + integer exactness
  toc_left       pinned: Theorem 2 (equals dense_left) + integer exactness
  map_values     pinned: Algorithm 3's claim (decoding the modified I equals the
                 element-wise op on the decoded batch), exact cases (c = 1, -1, 2),
                 squares of integers
  dense_plus     pinned: round trip to the CSR for c = 0, zeros become c,
                 integer sums in closed form
  layout_stats   pinned: hand count on the worked example (live set, depths)
  level_order    pinned: the worked example's level order derived by hand from
                 Table 4; invariants (parents first, depth steps of one, stable
                 within a depth, exactly the live set) and decoding through the new
                 numbering equal to Algorithm 6 on random tables
  physical_bytes parity unpinned (the paper prints sizes only in missing figures;
                 the formula of §3.2 is checked on the worked example by hand)
  dense_bytes, sparse_bytes, logical_bytes
                 pinned: hand counts on the worked example (12 pairs, |I| = 5,
                 |D| = 9); the byte layouts are a reading (the paper gives none)
  pack_physical, unpack_physical
                 pinned: the worked example's bytes derived by hand from Table 2's
                 I and D under the byte-layout reading, the width rule of §3.2 at
                 every byte boundary (its "max 4 needs 1 byte" example included),
                 round trips, size equal to physical_bytes, malformed inputs
  mgd_loss, mgd_dloss, mgd_step
                 pinned: central finite differences of the mean loss (the step is
                 h - lr * its gradient) for all three losses on random batches,
                 the paper's linear-regression gradient on the worked example by
                 hand, closed forms (lr = 0, one entry, logistic at r = 0, hinge
                 beyond the margin), an empty batch
  mlp_grad_scale pinned: at least |gradient| for every entry; at zero weights
                 the closed form (only the output layer's scales are nonzero, the
                 bias's being the mean of |1/C - [y = c]|)
  mlp_loss, mlp_step
                 pinned: central finite differences of the mean cross-entropy for
                 every parameter (softmax and single-sigmoid outputs), the first
                 layer's gradient equal to Theorem 2's left product on (I, D)
                 (toc_left), the closed form at zero weights, lr = 0, an empty batch
"""

from .toc_oracle import (  # noqa: F401
    TocInputError,
    canonicalize,
    encode,
    build_cprime,
    decode,
    densify,
    mlp_grad_scale,
    decoded_to_csr,
    dense_right,
    dense_left,
    toc_right,
    toc_left,
    map_values,
    dense_plus,
    MAP_SCALE,
    MAP_SQUARE,
    layout_stats,
    level_order,
    physical_bytes,
    dense_bytes,
    sparse_bytes,
    logical_bytes,
    pack_physical,
    unpack_physical,
    MGD_LINEAR,
    MGD_LOGISTIC,
    MGD_HINGE,
    mgd_loss,
    mgd_dloss,
    mgd_step,
    mlp_loss,
    mlp_step,
    f32_bits,
    bits_f32,
)
