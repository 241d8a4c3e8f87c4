"""Full-size parity for the benchmark workload (image-like MLP first layer: 40,000
mini-batches x 250 rows x 784 columns, k = 300), in the launch configuration
bench.py times: one upload of every batch, one launch of each op.

The oracle checks sampled batches one by one (products within 1e-5 * S, decode
bit-exact against the regenerated batch); properties that hold at any size are
checked on the whole output.
"""

import multiprocessing as mp
import os

import numpy as np
import pytest

import oracle as O
from workloads import CONFIGS, config_batches, config_W
from workloads.parallel import default_workers

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu, pytest.mark.slow]

CFG = "c3"
TOL = 1e-5


def _pool():
    ctx = "spawn" if torch.cuda.is_initialized() else "fork"
    return mp.get_context(ctx).Pool(default_workers())


@pytest.mark.timeout(1200)
def test_fullsize_bench_workload_sampled():
    import bench
    spec = CONFIGS[CFG]
    nb, k = spec["n_batches"], spec["k"]
    pool = _pool()
    try:
        w = bench.encode_workload(CFG, nb, pool)
    finally:
        pool.close()
        pool.join()
    bench.upload_workload(w, k)
    w.encs = None
    info = w.info
    assert info["n_batches"] == nb and info["n_rows"] == nb * spec["rows"]
    bench.run_ops(w)
    torch.cuda.synchronize()
    print(f"full size: {nb} batches, nnz {info['nnz']}, image {info['image_bytes']} B",
          flush=True)

    # properties of the whole decoded CSR
    rowptr = w.rowptr.cpu().numpy()
    assert rowptr[0] == 0 and rowptr[-1] == info["nnz"]
    assert np.all(np.diff(rowptr) >= 0)
    assert np.all(np.diff(rowptr) == 157)       # every row of this workload keeps 157 pixels
    assert torch.isfinite(w.R).all().item() and torch.isfinite(w.out).all().item()

    W = config_W(CFG, k).astype(np.float64)
    rng = np.random.default_rng(20240601)
    sample = sorted({0, 1, nb // 2, nb - 1, *rng.integers(0, nb, size=8).tolist()})
    rows, m = spec["rows"], spec["cols"]
    worst = 0.0
    for b in sample:
        B = config_batches(CFG, b, 1)
        n, rp, c, v = B.batch(0)
        r0 = b * rows
        canon = O.canonicalize(n, m, rp, c, v)
        # products
        R_ref, S = O.dense_right(canon, m, W)
        R = w.R[r0:r0 + n].cpu().numpy().astype(np.float64)
        err = np.abs(R - R_ref)
        assert np.all(err <= TOL * S), f"right mul, batch {b}"
        worst = max(worst, float(np.max(err / np.maximum(S, 1e-300))))
        G = w.G[r0:r0 + n].cpu().numpy()
        out_ref, S = O.dense_left(canon, m, G)
        out = w.out[b * m:(b + 1) * m].cpu().numpy().astype(np.float64)
        err = np.abs(out - out_ref)
        assert np.all(err <= TOL * S), f"left mul, batch {b}"
        worst = max(worst, float(np.max(err / np.maximum(S, 1e-300))))
        # decode, bit-exact against the regenerated batch
        p0, p1 = int(rowptr[r0]), int(rowptr[r0 + n])
        assert np.array_equal(rowptr[r0:r0 + n + 1] - p0, rp)
        assert np.array_equal(w.ccol[p0:p1].cpu().numpy(), c)
        assert np.array_equal(w.cval[p0:p1].cpu().numpy().view(np.uint32), v.view(np.uint32))
    print(f"sampled batches {sample}: max |err|/S = {worst:.3e}", flush=True)
