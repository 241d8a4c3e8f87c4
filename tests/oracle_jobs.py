"""Oracle work for GPU tests, run in worker processes: each job regenerates one
seeded batch of a workload and computes the oracle's fp64 products and decode.
Imports only the oracle and the input generators (never the HIP path)."""

import numpy as np

import oracle as O
from workloads import config_batches, config_G


def products(job):
    """job = (cfg, batch, W, k) -> (R_ref, S_R, out_ref, S_out, rowptr, col, val
    bits) of that batch of the workload, G being the workload's own seeded G rows
    and (rowptr, col, val) the canonical CSR that decoding must give back."""
    cfg, b, W, k = job
    B = config_batches(cfg, b, 1)
    n, rp, c, v = B.batch(0)
    rows = O.canonicalize(n, B.n_cols, rp, c, v)
    R, SR = O.dense_right(rows, B.n_cols, W)
    G = config_G(cfg, b, 1, k)
    out, SO = O.dense_left(rows, B.n_cols, G)
    # decode is lossless: the decoded CSR must equal the canonical input
    crp, cc, cv = O.decoded_to_csr(rows)
    return R, SR, out, SO, crp, cc, np.asarray(cv).view(np.uint32)
