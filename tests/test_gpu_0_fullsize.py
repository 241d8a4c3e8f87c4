"""Full-size parity in the launch configuration bench.py times: one upload of
every batch of a workload, one launch of each op over all of them.

* image-like MLP first layer: 40,000 mini-batches x 250 rows x 784 columns, k = 300
  (the benchmark workload);
* dense quantised features, wide hidden layer: 20,000 mini-batches x 250 rows x
  1,000 columns, k = 200 (a 145 GB image, uploaded in chunks through pinned
  staging buffers).

For the first, the image is also built on the device from the batches' physical
bytes (section 3.2) and must equal the host-built one byte for byte.

The oracle checks sampled batches one by one (products within 1e-5 * S, decode
bit-exact against the regenerated batch); properties that hold at any size are
checked on the whole output.
"""

import gc
import multiprocessing as mp

import numpy as np
import pytest

import oracle as O
from workloads import CONFIGS, config_batches, config_W
from workloads.parallel import default_workers

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu, pytest.mark.slow]

TOL = 1e-5
# every row of these workloads keeps the same number of entries
ROW_NNZ = {"c3": 157, "c4": 1000}


def _pool():
    ctx = "spawn" if torch.cuda.is_initialized() else "fork"
    return mp.get_context(ctx).Pool(default_workers())


@pytest.mark.timeout(1200)
@pytest.mark.parametrize("cfg", ["c3", "c4"])
def test_fullsize_sampled(cfg):
    import bench
    spec = CONFIGS[cfg]
    nb, k = spec["n_batches"], spec["k"]
    print(f"full size {cfg}: {nb} batches, k = {k}", flush=True)
    pool = _pool()
    try:
        w = bench.encode_workload(cfg, nb, pool)
    finally:
        pool.close()
        pool.join()
    try:
        _check_workload(bench, w, cfg, spec, nb, k)
    finally:
        w.encs = None
        del w
        gc.collect()
        torch.cuda.empty_cache()


def _check_workload(bench, w, cfg, spec, nb, k):
    bench.upload_workload(w, k)
    packed = bench.pack_all(w) if cfg == "c3" else None
    w.encs = None
    info = w.info
    assert info["n_batches"] == nb and info["n_rows"] == nb * spec["rows"]
    bench.run_ops(w)
    torch.cuda.synchronize()
    print(f"full size {cfg}: nnz {info['nnz']}, image {info['image_bytes']} B", flush=True)

    # properties of the whole decoded CSR and of the products
    rowptr = w.rowptr.cpu().numpy()
    assert rowptr[0] == 0 and rowptr[-1] == info["nnz"]
    assert np.all(np.diff(rowptr) == ROW_NNZ[cfg])
    assert torch.isfinite(w.R).all().item() and torch.isfinite(w.out).all().item()

    W = config_W(cfg, k).astype(np.float64)
    rng = np.random.default_rng(20240601 + spec["cid"])
    sample = sorted({0, 1, nb // 2, nb - 1, *rng.integers(0, nb, size=8).tolist()})
    rows, m = spec["rows"], spec["cols"]
    worst = 0.0
    for b in sample:
        B = config_batches(cfg, b, 1)
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
    print(f"{cfg} sampled batches {sample}: max |err|/S = {worst:.3e}", flush=True)
    if packed is not None:
        ing = bench.time_ingest(w, packed)
        print(f"{cfg} device ingest: {ing}", flush=True)
        assert ing["identical_to_host_image"]
