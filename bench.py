#!/usr/bin/env python3
"""Benchmark of the TOC hot path on one MI355X.

One step = A.W (right multiplication), G^T.A (left multiplication) and decode to
CSR over every mini-batch of a workload, with the compressed image, W and G
already resident in HBM.  Encoding and upload happen once before timing, as the
paper excludes compression time from training time.

Prints one JSON line (see --help for the options).
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

HBM_PEAK = 8.0e12                     # bytes/s, MI355X HBM3E
# MI355X's published fp32 vector peak: 256 CUs x 4 SIMDs x 16 lanes x 2 FMAs per lane
# and clock (packed FP32) x 2 flops x 2.4 GHz
FP32_PEAK = 256 * 4 * 16 * 2 * 2 * 2.4e9
# the issue rate of one (non-packed) FMA per lane and clock: the ceiling of code
# built without packed-FP32 instructions, as this library is
FP32_NONPACKED_PEAK = FP32_PEAK / 2
# workloads whose batches are dense enough that the CPU baseline multiplies the
# densified batch (fp64 numpy matmul); the others use the oracle's sparse products
DENSE_CPU = ("c1", "c3", "c4")
METRIC = "uncompressed nnz/s for TOC A·W and Gᵀ·A; % HBM peak on compressed bytes"
HERE = os.path.dirname(os.path.abspath(__file__))


def log(msg):
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


# ---------------------------------------------------------------------------
# CPU baseline: the oracle, timed on a sample of the workload's batches.  Per batch,
# separately: the products A.W and G^T.A in fp64 on the decoded batch (dense
# workloads: the densified batch times W and its transpose times G, numpy matmuls;
# sparse ones: the oracle's sparse products), the oracle's decode (Algorithm 6) and
# its encode (Algorithm 1).  The products are the baseline's value.
# ---------------------------------------------------------------------------
def _oracle_batch(args):
    cfg, b, k = args
    import oracle as O
    from threadpoolctl import threadpool_limits
    from workloads import config_batches, config_G, config_W
    B = config_batches(cfg, b, 1)
    n, rp, c, v = B.batch(0)
    W = config_W(cfg, k).astype(np.float64)
    G = config_G(cfg, b, 1, k).astype(np.float64)
    rows = O.canonicalize(n, B.n_cols, rp, c, v)
    with threadpool_limits(limits=1):                 # one core per batch
        t0 = time.perf_counter()
        I, D, _ = O.encode(rows)
        t_enc = time.perf_counter() - t0
        t0 = time.perf_counter()
        dec = O.decode(I, D)
        O.decoded_to_csr(dec)
        t_dec = time.perf_counter() - t0
        t0 = time.perf_counter()
        if cfg in DENSE_CPU:
            A = O.densify(dec, B.n_cols)
            _ = A @ W
            _ = A.T @ G
        else:
            O.dense_right(dec, B.n_cols, W)
            O.dense_left(dec, B.n_cols, G)
        t_prod = time.perf_counter() - t0
    return t_prod, t_dec, t_enc, int(B.nnz)


def _cpu_rates(res, cores):
    """nnz/s of each part with `cores` batches at a time: nnz over the summed
    per-batch times divided by the cores."""
    nnz = sum(r[3] for r in res)
    t = [sum(r[i] for r in res) for i in range(3)]
    return {name: nnz * cores / max(t[i], 1e-12)
            for i, name in enumerate(("products", "decode", "encode"))}, t


def cpu_baseline(pool, workers, cfg, nb, k, budget_s):
    t1 = sum(_oracle_batch((cfg, 0, k))[:3])
    n_sample = int(min(max(workers, round(budget_s * workers / max(t1, 1e-3))), nb, 4000))
    ids = sorted(set(np.linspace(0, nb - 1, n_sample).astype(int).tolist()))
    t0 = time.perf_counter()
    res = pool.map(_oracle_batch, [(cfg, b, k) for b in ids])
    wall = time.perf_counter() - t0
    rates, t = _cpu_rates(res, workers)
    how = ("the densified batch (fp64 numpy matmuls A @ W and A.T @ G)" if cfg in DENSE_CPU
           else "the decoded batch (the oracle's fp64 sparse products)")
    return {
        "value": rates["products"],
        "unit": "nnz/s",
        "cores": workers,
        "kind": "oracle",
        "sample": f"{len(ids)} of {nb} mini-batches evenly spaced over the workload, one "
                  f"batch per core at a time on {workers} worker processes ({wall:.1f} s "
                  f"wall); value = A.W + G^T.A in fp64 on {how}, nnz over the summed "
                  f"per-batch product times ({t[0]:.1f} s) / {workers} cores; the oracle's "
                  f"decode (Algorithm 6, {t[1]:.1f} s) and encode (Algorithm 1, {t[2]:.1f} "
                  f"s) are timed apart in `parts`",
        "parts_nnz_per_s": rates,
    }


def cpu_baseline_single(cfg, nb, k, budget_s):
    """The same oracle work on one core, in this process: batches evenly spaced
    over the workload until about budget_s seconds of it are done."""
    res = []
    ids = np.linspace(0, nb - 1, min(nb, 400)).astype(int).tolist()
    for b in ids:
        res.append(_oracle_batch((cfg, b, k)))
        if sum(sum(r[:3]) for r in res) >= budget_s:
            break
    rates, t = _cpu_rates(res, 1)
    return {"value": rates["products"], "unit": "nnz/s", "cores": 1, "kind": "oracle",
            "sample": f"{len(res)} mini-batches evenly spaced over the workload, one process, "
                      f"BLAS on one thread; products {t[0]:.2f} s, decode {t[1]:.2f} s, "
                      f"encode {t[2]:.2f} s",
            "parts_nnz_per_s": rates}


def host_cpu():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


# ---------------------------------------------------------------------------
# Workload preparation: generate (process pool) -> encode (C++ threads) -> upload
# ---------------------------------------------------------------------------
class Workload:
    pass


def encode_workload(cfg, nb, pool, chunk=400, keep_batches=0):
    """Generates and host-encodes the workload; keeps the CSR of the first
    keep_batches batches (w.kept) for the device encoder's measurement."""
    import paper_1702_06943_amd as T
    from workloads.parallel import iter_chunks
    w = Workload()
    w.cfg, w.nb = cfg, nb
    w.encs, w.nnz, w.rows, w.kept = [], 0, 0, []
    t0 = time.perf_counter()
    last = t0
    for part in iter_chunks(cfg, nb, 0, chunk, pool):
        if len(w.encs) < keep_batches:
            w.kept.append(part)
        w.encs.extend(T.toc_encode_batches(part.n_rows, part.n_cols, part.rowptr, part.col,
                                           part.val))
        w.nnz += part.nnz
        w.rows += int(part.n_rows.sum())
        w.n_cols = part.n_cols
        if time.perf_counter() - last > 10 or len(w.encs) == nb:
            log(f"generated+encoded {len(w.encs)}/{nb} batches "
                f"({time.perf_counter() - t0:.1f} s)")
            last = time.perf_counter()
    w.encode_s = time.perf_counter() - t0
    return w


def upload_workload(w, k, device="cuda:0", seed_G=None):
    import torch
    import paper_1702_06943_amd as T
    from workloads import CONFIGS, config_W, dense_normal_device, SEED
    spec = CONFIGS[w.cfg]
    t0 = time.perf_counter()
    size = T.toc_upload_size(w.encs)
    # zeroed, so that the padding between arrays is defined (the device-built
    # image is compared with this one byte for byte)
    w.buf = torch.zeros(size, dtype=torch.uint8, device=device)
    w.dev = T.toc_upload(w.encs, w.buf)
    w.upload_s = time.perf_counter() - t0
    w.info = T.toc_dev_info_get(w.dev)
    log(f"uploaded image: {size / 1e9:.2f} GB in {w.upload_s:.1f} s")
    w.k = k
    w.W = torch.from_numpy(config_W(w.cfg, k)).to(device)
    seed = SEED * 16 + spec["cid"] if seed_G is None else seed_G
    w.G = dense_normal_device((w.info["n_rows"], k), 1.0, seed, device)
    w.R = torch.empty((w.info["n_rows"], k), device=device)
    w.out = torch.empty((w.info["n_batches"] * w.info["n_cols"], k), device=device)
    w.rowptr = torch.empty(w.info["n_rows"] + 1, dtype=torch.int64, device=device)
    w.ccol = torch.empty(max(w.info["nnz"], 1), dtype=torch.int32, device=device)[:w.info["nnz"]]
    w.cval = torch.empty(max(w.info["nnz"], 1), dtype=torch.float32, device=device)[:w.info["nnz"]]
    ws_r, _ = T.toc_workspace_size(w.dev, T.TOC_OP_RIGHT, k)
    ws_l, _ = T.toc_workspace_size(w.dev, T.TOC_OP_LEFT, k)
    w.ws_r = torch.empty(max(ws_r // 4, 1), device=device) if ws_r else None
    w.ws_l = torch.empty(max(ws_l // 4, 1), device=device) if ws_l else None
    torch.cuda.synchronize()
    return w


def run_ops(w, which=("right", "left", "decode")):
    import paper_1702_06943_amd as T
    if "right" in which:
        T.toc_right_mul(w.dev, w.W, w.R, w.ws_r)
    if "left" in which:
        T.toc_left_mul(w.dev, w.G, w.out, False, w.ws_l)
    if "decode" in which:
        T.toc_decode_csr(w.dev, w.rowptr, w.ccol, w.cval)


def time_ops(w, steps, warmup, stream, names=("right", "left", "decode")):
    """warmup untimed steps, then `steps` timed ones; events around each op on the
    stream the kernels run on.  Returns (per-op mean ms, mean step ms, wall s)."""
    import torch
    for _ in range(warmup):
        run_ops(w, names)
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(names) + 1)]
          for _ in range(steps)]
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    for s in range(steps):
        ev[s][0].record(stream)
        for i, op in enumerate(names):
            run_ops(w, (op,))
            ev[s][i + 1].record(stream)
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    op_ms = {op: float(np.mean([ev[s][i].elapsed_time(ev[s][i + 1]) for s in range(steps)]))
             for i, op in enumerate(names)}
    step_ms = float(np.mean([ev[s][0].elapsed_time(ev[s][len(names)]) for s in range(steps)]))
    return op_ms, step_ms, t_wall


def op_bytes_flops(info, k):
    """Algorithmic dense bytes (beyond the canonical compressed bytes) and flops of
    each op over the whole workload (one launch of each op)."""
    m, n_rows, nnz = info["n_cols"], info["n_rows"], info["nnz"]
    dense = {
        "right": 4 * m * k + 4 * n_rows * k,                         # W once, R
        "left": 4 * n_rows * k + 4 * info["n_batches"] * m * k,      # G, out
        "decode": 8 * (n_rows + 1) + 8 * nnz,                        # rowptr, col+val
    }
    flops = {
        "right": 2.0 * k * (info["n_deep"] + info["n_codes"]),
        "left": 2.0 * k * (info["n_codes"] + info["n_stored"] + info["n_deep"]),
        "decode": 0.0,
    }
    return dense, flops


def op_report(info, k, op_ms, copy_bw=None):
    """Per op: time, uncompressed nnz/s, the literal fraction of the HBM peak on
    the canonical compressed bytes and the fraction on the whole op's bytes."""
    dense, flops = op_bytes_flops(info, k)
    canon, nnz = info["canon_bytes"], info["nnz"]
    ops = {}
    for op, ms in op_ms.items():
        t = ms / 1e3
        ops[op] = {
            "ms": round(ms, 4),
            "nnz_per_s": nnz / t,
            "hbm_frac_compressed": canon / t / HBM_PEAK,
            "hbm_frac_whole_op": (canon + dense[op]) / t / HBM_PEAK,
            "tflops": flops[op] / t / 1e12,
        }
        if copy_bw:
            ops[op]["frac_of_measured_copy_compressed"] = canon / t / copy_bw
            ops[op]["frac_of_measured_copy_whole_op"] = (canon + dense[op]) / t / copy_bw
    return ops


def time_k1_workloads(ws, steps, warmup, stream):
    """The k = 1 workloads (each pre-encoded before the GPU was touched): upload,
    time right, left and decode like the main step, report, free."""
    import torch
    out = {}
    for w in ws:
        upload_workload(w, 1)
        w.encs = None
        op_ms, step_ms, _ = time_ops(w, steps, warmup, stream)
        ops = op_report(w.info, 1, op_ms)
        out[w.cfg] = {"batches": w.nb, "nnz": w.info["nnz"], "canon_bytes": w.info["canon_bytes"],
                      "image_bytes": w.info["image_bytes"], "step_ms": round(step_ms, 4),
                      "nnz_per_s": w.info["nnz"] / (step_ms / 1e3), "ops": ops,
                      "upload_s": round(w.upload_s, 2), "encode_s": round(w.encode_s, 2)}
        log(f"{w.cfg} (k = 1, {w.nb} batches): step {step_ms:.3f} ms; " + ", ".join(
            f"{o} {v['ms']:.3f} ms ({v['hbm_frac_compressed']:.1%} literal, "
            f"{v['hbm_frac_whole_op']:.1%} whole-op)" for o, v in ops.items()))
        for a in ("buf", "dev", "W", "G", "R", "out", "rowptr", "ccol", "cval", "ws_r", "ws_l"):
            setattr(w, a, None)
        torch.cuda.empty_cache()
    return out


def time_elementwise(w, stream, reps=3):
    """The element-wise operations on the same resident image, outside the step:
    toc_map_values with c = 1 (the matrix is unchanged) and toc_decode_dense with
    c = 0 into a dense n_rows x n_cols block when it fits in free memory.  HBM
    fractions use algorithmic bytes: 4-byte read and write of every key value and
    its position copy; the canonical bytes read plus the dense block written."""
    import torch
    import paper_1702_06943_amd as T
    info = w.info
    res = {}
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
    T.toc_map_values(w.dev, T.TOC_MAP_SCALE, 1.0)
    ev[0].record(stream)
    for i in range(reps):
        T.toc_map_values(w.dev, T.TOC_MAP_SCALE, 1.0)
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    ms = float(np.mean([ev[i].elapsed_time(ev[i + 1]) for i in range(reps)]))
    b = 16.0 * info["n_stored"]
    res["map_values"] = {"ms": round(ms, 4), "bytes": b, "GB/s": b / ms / 1e6,
                         "hbm_frac": b / (ms / 1e3) / HBM_PEAK}
    dense_bytes = 4 * info["n_rows"] * info["n_cols"]
    free, _ = torch.cuda.mem_get_info()
    if dense_bytes + (1 << 30) < free:
        A = torch.empty((info["n_rows"], info["n_cols"]), dtype=torch.float32, device="cuda:0")
        T.toc_decode_dense(w.dev, A, 0.0)
        ev[0].record(stream)
        for i in range(reps):
            T.toc_decode_dense(w.dev, A, 0.0)
            ev[i + 1].record(stream)
        torch.cuda.synchronize()
        ms = float(np.mean([ev[i].elapsed_time(ev[i + 1]) for i in range(reps)]))
        b = float(info["canon_bytes"] + dense_bytes)
        res["decode_dense"] = {"ms": round(ms, 4), "bytes": b, "GB/s": b / ms / 1e6,
                               "hbm_frac": b / (ms / 1e3) / HBM_PEAK}
        del A
        torch.cuda.empty_cache()
    else:
        res["decode_dense"] = None
    log("element-wise: " + ", ".join(f"{k} {v['ms']:.3f} ms ({v['hbm_frac']:.1%} of HBM peak)"
                                     for k, v in res.items() if v))
    return res


def pack_sample(w, n):
    """Physical encodings (section 3.2) of n batches spread evenly over the workload,
    packed on the host from the encodings before they are dropped."""
    import paper_1702_06943_amd as T
    if n <= 0:
        return None
    idx = np.linspace(0, len(w.encs) - 1, min(n, len(w.encs))).astype(np.int64)
    t0 = time.perf_counter()
    blobs = [T.toc_enc_pack(w.encs[i]) for i in idx]
    return {"blobs": blobs, "pack_s": time.perf_counter() - t0, "cfg": w.cfg, "n_cols": w.n_cols}


def _host_map(fn, items, threads=16):
    """fn over items on host threads (the library's calls release the GIL)."""
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(max_workers=threads) as ex:
        return list(ex.map(fn, items, chunksize=64))


def pack_all(w):
    """Physical encodings (section 3.2) of every batch, packed on the host."""
    import paper_1702_06943_amd as T
    t0 = time.perf_counter()
    blobs = _host_map(T.toc_enc_pack, w.encs)
    infos = _host_map(T.toc_phys_info_get, blobs)
    off = np.concatenate([[0], np.cumsum([len(b) for b in blobs])]).astype(np.int64)
    cat = np.concatenate(blobs + [np.zeros(1, np.uint8)])
    return {"cat": cat, "off": off, "infos": infos, "pack_s": time.perf_counter() - t0}


def time_ingest(w, packed, ws_gib=8):
    """The whole workload's image built on the device from its physical bytes
    (toc_ingest_plan + toc_ingest_build), after copying only those bytes to HBM; the
    result is compared byte for byte with the image toc_upload built on the host."""
    import torch
    import paper_1702_06943_amd as T
    dev = "cuda:0"
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    d_blobs = torch.from_numpy(packed["cat"]).to(dev)
    torch.cuda.synchronize()
    h2d_s = time.perf_counter() - t0
    full, least = T.toc_ingest_workspace_size(packed["infos"], w.n_cols)
    ws_bytes = max(least, min(full, ws_gib << 30))
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    t0 = time.perf_counter()
    size, idev = T.toc_ingest_plan(d_blobs, packed["off"], packed["infos"], w.n_cols, ws)
    plan_s = time.perf_counter() - t0
    buf = torch.empty(size, dtype=torch.uint8, device=dev)
    t0 = time.perf_counter()
    T.toc_ingest_build(idev, d_blobs, packed["off"], buf, ws)
    build_s = time.perf_counter() - t0
    same = size == w.info["image_bytes"]
    step = 1 << 30
    for a in range(0, size if same else 0, step):
        bsz = min(step, size - a)
        if not torch.equal(buf[a:a + bsz], w.buf[a:a + bsz]):
            same = False
            break
    del buf, ws, d_blobs, idev
    torch.cuda.empty_cache()
    phys = int(packed["off"][-1])
    log(f"device ingest: {phys / 1e9:.2f} GB of physical bytes -> {size / 1e9:.2f} GB image: "
        f"copy {h2d_s:.2f} s, plan {plan_s:.2f} s, build {build_s:.2f} s, "
        f"identical to the host-built image: {same}")
    return {"phys_bytes": phys, "image_bytes": int(size), "canon_bytes": w.info["canon_bytes"],
            "pack_s": round(packed["pack_s"], 2), "h2d_s": round(h2d_s, 3),
            "plan_s": round(plan_s, 3), "build_s": round(build_s, 3),
            "ws_bytes": int(ws_bytes), "identical_to_host_image": bool(same),
            "host_path_s": round(w.encode_s + w.upload_s, 2)}


def time_cprime(sample, stream, reps=3):
    """toc_cprime_build over the sampled batches' physical bytes, resident in HBM.
    Algorithmic bytes: the blobs read once plus 16 bytes written per node."""
    import torch
    import paper_1702_06943_amd as T
    blobs = sample["blobs"]
    infos = [T.toc_phys_info_get(b) for b in blobs]
    blob_off = np.concatenate([[0], np.cumsum([len(b) for b in blobs])]).astype(np.int64)
    node_off = np.concatenate([[0], np.cumsum([i["n_nodes"] for i in infos])]).astype(np.int64)
    n = int(node_off[-1])
    dev = "cuda:0"
    d_blobs = torch.from_numpy(np.concatenate(blobs)).to(dev)
    outs = [torch.empty(n, dtype=torch.int32, device=dev) for _ in range(4)]
    status = torch.empty(len(blobs), dtype=torch.int32, device=dev)
    ws = torch.empty(T.toc_cprime_workspace_size(len(blobs), n), dtype=torch.uint8, device=dev)
    max_rows = max(i["n_rows"] for i in infos)
    n_cols = sample["n_cols"]

    def run():
        T.toc_cprime_build(d_blobs, blob_off, node_off, max_rows, n_cols, *outs, status, ws)

    run()
    torch.cuda.synchronize()
    ok = bool((status == 0).all().item())
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * reps)]
    for i in range(reps):
        ev[2 * i].record(stream)
        run()
        ev[2 * i + 1].record(stream)
    torch.cuda.synchronize()
    ms = float(np.mean([ev[2 * i].elapsed_time(ev[2 * i + 1]) for i in range(reps)]))
    # then the live codes in level order from that tree (toc_level_build)
    d_off = np.concatenate([[0], np.cumsum([i["n_codes"] for i in infos])]).astype(np.int64)
    max_levels = 64
    lv = [torch.empty(n, dtype=torch.int32, device=dev) for _ in range(4)]
    level = torch.empty(len(blobs) * (max_levels + 1), dtype=torch.int32, device=dev)
    lD = torch.empty(max(int(d_off[-1]), 1), dtype=torch.int32, device=dev)
    counts = torch.empty(2 * len(blobs), dtype=torch.int64, device=dev)
    lst = torch.empty(len(blobs), dtype=torch.int32, device=dev)
    ws2 = torch.empty(T.toc_level_workspace_size(len(blobs), n), dtype=torch.uint8, device=dev)

    def run_level():
        T.toc_level_build(d_blobs, blob_off, node_off, d_off, max_levels, status, *outs, *lv,
                          level, lD, counts, lst, ws2)

    run_level()
    torch.cuda.synchronize()
    lok = bool((lst == 0).all().item())
    n_live = int(counts.view(-1, 2)[:, 0].sum().item())
    for i in range(reps):
        ev[2 * i].record(stream)
        run_level()
        ev[2 * i + 1].record(stream)
    torch.cuda.synchronize()
    lms = float(np.mean([ev[2 * i].elapsed_time(ev[2 * i + 1]) for i in range(reps)]))
    # and A.w (k = 1) from that level order (toc_level_right_mul): bytes to product
    # without any host pass
    from workloads import config_W
    row_off = np.concatenate([[0], np.cumsum([i["n_rows"] for i in infos])]).astype(np.int64)
    max_live = int(counts.view(-1, 2)[:, 0].max().item())
    wv = torch.from_numpy(np.ascontiguousarray(config_W(sample["cfg"], 1)[:, 0])).to(dev)
    rv = torch.empty(max(int(row_off[-1]), 1), device=dev)
    rst = torch.empty(len(blobs), dtype=torch.int32, device=dev)
    ws3 = torch.empty(32 * (len(blobs) + 1), dtype=torch.uint8, device=dev)

    def run_right():
        T.toc_level_right_mul(d_blobs, blob_off, node_off, d_off, row_off, max_levels, max_live,
                              lst, counts, level, lv[0], lv[1], lv[2], lD, wv, rv, rst, ws3)

    rms = None
    try:
        run_right()
        torch.cuda.synchronize()
        rok = bool((rst == 0).all().item())
        for i in range(reps):
            ev[2 * i].record(stream)
            run_right()
            ev[2 * i + 1].record(stream)
        torch.cuda.synchronize()
        rms = float(np.mean([ev[2 * i].elapsed_time(ev[2 * i + 1]) for i in range(reps)]))
    except T.TocError as e:
        log(f"product from the level order skipped: {e}")
        rok = False
    # algorithmic bytes: the tree read once (16 B per node), D read from the blobs
    # and written renumbered, 16 B per live code and the level offsets written
    lb = float(16 * n + 8 * int(d_off[-1]) + 16 * n_live + 4 * level.numel())
    b = float(blob_off[-1] + 16 * n)
    res = {"batches": len(blobs), "nodes": n, "blob_bytes": int(blob_off[-1]), "ms": round(ms, 4),
           "nodes_per_s": n / (ms / 1e3), "GB/s": b / ms / 1e6,
           "hbm_frac": b / (ms / 1e3) / HBM_PEAK, "status_ok": ok,
           "host_pack_s": round(sample["pack_s"], 3),
           "level_order": {"ms": round(lms, 4), "live_codes": n_live,
                           "hbm_frac": lb / (lms / 1e3) / HBM_PEAK, "status_ok": lok},
           "ingest_ms": round(ms + lms, 4),
           "right_k1_from_level_order": None if rms is None else
           {"ms": round(rms, 4), "status_ok": rok,
            "bytes_to_product_ms": round(ms + lms + rms, 4)}}
    log(f"C' build from physical bytes: {len(blobs)} batches, {n} nodes, {ms:.3f} ms "
        f"({res['hbm_frac']:.1%} of HBM peak on algorithmic bytes), status ok: {ok}")
    log(f"level order from that tree: {lms:.3f} ms ({res['level_order']['hbm_frac']:.1%} of "
        f"HBM peak on algorithmic bytes), {n_live} live codes, status ok: {lok}")
    if rms is not None:
        log(f"A.w (k = 1) from that level order: {rms:.3f} ms; bytes to product "
            f"{ms + lms + rms:.3f} ms, status ok: {rok}")
    del d_blobs, outs, status, ws, lv, level, lD, counts, lst, ws2, wv, rv, rst, ws3
    torch.cuda.empty_cache()
    return res


def time_mgd(w, stream, lr=0.1):
    """One epoch of mini-batch gradient descent for logistic regression (k = 1) over
    every batch of the resident image (each step depends on the previous one), with
    seeded labels of +-1 and h = 0 at the start: with the steps split over many
    workgroups (toc_mgd_epoch_split, two launches a step; the reported figure), and
    in one launch of one workgroup (toc_mgd_epoch)."""
    import torch
    import paper_1702_06943_amd as T
    info = w.info
    gen = torch.Generator(device="cuda:0")
    gen.manual_seed(1702)
    y = (torch.randint(0, 2, (info["n_rows"],), generator=gen, device="cuda:0") * 2 - 1).float()
    h = torch.zeros(info["n_cols"], device="cuda:0")
    ws = torch.empty(T.toc_mgd_workspace_size(w.dev), dtype=torch.uint8, device="cuda:0")
    runs = {"split": lambda **kw: T.toc_mgd_epoch_split(w.dev, y, h, T.TOC_MGD_LOGISTIC, lr, ws, **kw),
            "one": lambda **kw: T.toc_mgd_epoch(w.dev, y, h, T.TOC_MGD_LOGISTIC, lr, **kw)}
    ms = {}
    for kind, run in runs.items():
        try:
            run(b0=0, n_batches=1)
        except T.TocError as e:
            log(f"MGD epoch ({kind}) skipped: {e}")
            continue
        h.zero_()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        ev[0].record(stream)
        run()
        ev[1].record(stream)
        torch.cuda.synchronize()
        ms[kind] = ev[0].elapsed_time(ev[1])
        if not bool(torch.isfinite(h).all().item()):
            ms[kind] = None
    if not ms.get("split"):
        return None
    t = ms["split"]
    res = {"loss": "logistic", "batches": info["n_batches"], "ms": round(t, 3),
           "us_per_step": t / info["n_batches"] * 1e3,
           "batches_per_s": info["n_batches"] / (t / 1e3),
           "nnz_per_s": info["nnz"] / (t / 1e3), "model_finite": True,
           "single_workgroup_ms": round(ms["one"], 3) if ms.get("one") else None}
    log(f"MGD epoch (logistic, {info['n_batches']} steps, split over workgroups): {t:.1f} ms, "
        f"{res['us_per_step']:.1f} us/step; one workgroup: "
        f"{ms.get('one') or float('nan'):.1f} ms")
    return res


def variant_sizes(infos, n_cols):
    """Bytes of the ablation study's TOC variants (section 5.2) summed over the
    batches, from the encoder's counts: DEN 4 n m; sparse encoding 8 nnz + 4 (n + 1);
    logical encoding 8 |I| + 4 |D| + 4 (n + 1); TOC_FULL the physical encoding of
    section 3.2.  Ratios are DEN over each."""
    tot = {"dense": 0, "sparse": 0, "logical": 0, "full": 0}
    for i in infos:
        n = i["n_rows"]
        tot["dense"] += 4 * n * n_cols
        tot["sparse"] += 8 * i["nnz"] + 4 * (n + 1)
        tot["logical"] += 8 * i["n_first"] + 4 * i["n_codes"] + 4 * (n + 1)
        tot["full"] += i["phys_bytes"]
    out = {f"{k}_bytes": v for k, v in tot.items()}
    for k in ("sparse", "logical", "full"):
        out[f"{k}_ratio"] = tot["dense"] / tot[k] if tot[k] else None
    return out


def time_encode_device(w, stream, reps=3):
    """toc_encode_device (Algorithm 1 on the GPU) over the kept batches' CSR,
    resident in HBM; counts checked against the host encoder's for every batch,
    whose own time on the same batches (all host threads) is reported beside it.
    Algorithmic bytes: the CSR read once, I, D and the tuple offsets written once."""
    import torch
    import paper_1702_06943_amd as T
    from workloads import Batches
    if not w.kept:
        return None
    B = Batches.concat(w.kept)
    nb = B.n_batches
    t0 = time.perf_counter()
    T.toc_encode_batches(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    host_s = time.perf_counter() - t0
    dev = "cuda:0"
    max_nnz = int(np.diff(B.rowptr[B.row_off]).max())
    d_rp = torch.from_numpy(B.rowptr).to(dev)
    d_col = torch.from_numpy(B.col).to(dev)
    d_val = torch.from_numpy(B.val).to(dev)
    nnz = int(B.col.size)
    I_col = torch.empty(max(nnz, 1), dtype=torch.int32, device=dev)
    I_val = torch.empty(max(nnz, 1), device=dev)
    D = torch.empty(max(nnz, 1), dtype=torch.int32, device=dev)
    D_rp = torch.empty(int(B.n_rows.sum()) + nb, dtype=torch.int64, device=dev)
    counts = torch.empty(4 * nb, dtype=torch.int64, device=dev)
    status = torch.empty(nb, dtype=torch.int32, device=dev)
    ws = torch.empty(max(T.toc_encode_device_workspace_size(nb, max_nnz), 1), dtype=torch.uint8,
                     device=dev)

    def run():
        T.toc_encode_device(B.n_rows, B.n_cols, d_rp, d_col, d_val, max_nnz, I_col, I_val, D,
                            D_rp, counts, status, ws)

    run()
    torch.cuda.synchronize()
    c = counts.cpu().numpy().reshape(nb, 4)
    ok = bool((status.cpu().numpy() == 0).all())
    infos = [T.toc_enc_info_get(e) for e in w.encs[:nb]]
    same = ok and all((c[b, 0], c[b, 1], c[b, 2]) == (infos[b]["n_first"], infos[b]["n_codes"],
                                                      infos[b]["n_nodes"]) for b in range(nb))
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * reps)]
    for i in range(reps):
        ev[2 * i].record(stream)
        run()
        ev[2 * i + 1].record(stream)
    torch.cuda.synchronize()
    ms = float(np.median([ev[2 * i].elapsed_time(ev[2 * i + 1]) for i in range(reps)]))
    n_first, n_codes = int(c[:, 0].sum()), int(c[:, 1].sum())
    b = 8.0 * (B.rowptr.size + nnz) + 8 * n_first + 4 * n_codes + 8 * (int(B.n_rows.sum()) + nb)
    res = {"batches": nb, "nnz": nnz, "ms": round(ms, 3), "nnz_per_s": nnz / (ms / 1e3),
           "hbm_frac": b / (ms / 1e3) / HBM_PEAK, "counts_equal_host": same,
           "host_encoder_ms": round(host_s * 1e3, 1),
           "host_encoder_nnz_per_s": nnz / host_s, "speedup_vs_host": host_s * 1e3 / ms,
           "workspace_bytes": int(ws.numel())}
    log(f"device encode: {nb} batches, {ms:.2f} ms ({res['nnz_per_s']:.3e} nnz/s); host "
        f"encoder on the same batches {host_s * 1e3:.1f} ms; counts equal: {same}")
    del d_rp, d_col, d_val, I_col, I_val, D, D_rp, counts, status, ws
    torch.cuda.empty_cache()
    return res


def time_mlp(w, stream, n_steps, h1=200, h2=50, n_out=10, lr=0.1):
    """n_steps mini-batch gradient descent steps of section 5.1's network (hidden
    layers of h1 and h2 sigmoid units, a softmax over n_out classes, cross-entropy)
    on the first batches of the resident image, in one toc_mlp_epoch call, with
    seeded labels and weights."""
    import torch
    import paper_1702_06943_amd as T
    info = w.info
    n_steps = min(n_steps, info["n_batches"])
    if n_steps <= 0:
        return None
    gen = torch.Generator(device="cuda:0")
    gen.manual_seed(5101)
    m = info["n_cols"]
    labels = torch.randint(0, n_out, (info["n_rows"],), generator=gen, device="cuda:0",
                           dtype=torch.int32)
    scale1 = 1.0 / max(1.0, float(info["nnz"]) / info["n_rows"]) ** 0.5 / 100.0
    p = {"W1": torch.randn((m, h1), generator=gen, device="cuda:0") * scale1,
         "b1": torch.zeros(h1, device="cuda:0"),
         "W2": torch.randn((h1, h2), generator=gen, device="cuda:0") * (1.0 / h1 ** 0.5),
         "b2": torch.zeros(h2, device="cuda:0"),
         "W3": torch.randn((h2, n_out), generator=gen, device="cuda:0") * (1.0 / h2 ** 0.5),
         "b3": torch.zeros(n_out, device="cuda:0")}
    ws = torch.empty(max(T.toc_mlp_workspace_size(w.dev, h1, h2, n_out), 16), dtype=torch.uint8,
                     device="cuda:0")
    try:
        T.toc_mlp_epoch(w.dev, p, labels, lr, ws, b0=0, n_batches=1)
    except T.TocError as e:
        log(f"NN steps skipped: {e}")
        return None
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    ev[0].record(stream)
    T.toc_mlp_epoch(w.dev, p, labels, lr, ws, b0=1, n_batches=n_steps)
    ev[1].record(stream)
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[1])
    ok = all(bool(torch.isfinite(t).all().item()) for t in p.values())
    res = {"layers": [m, h1, h2, n_out], "steps": n_steps, "ms": round(ms, 3),
           "steps_per_s": n_steps / (ms / 1e3), "ms_per_step": ms / n_steps,
           "epoch_s_extrapolated": info["n_batches"] * ms / n_steps / 1e3,
           "model_finite": ok}
    log(f"NN MGD ({m}-{h1}-{h2}-{n_out}, {n_steps} steps): {ms:.1f} ms, "
        f"{res['steps_per_s']:.0f} steps/s")
    return res


def measured_copy_bandwidth(stream, mib=4096, reps=5):
    """Bytes moved per second (read + write) by a plain device-to-device copy of
    `mib` MiB, the best of `reps`: the HBM rate a streaming kernel can reach here."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, device="cuda:0")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    best = float("inf")
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        dst.copy_(src)
        e1.record(stream)
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1))
    del src, dst
    torch.cuda.empty_cache()
    return 2.0 * n * 4 / (best / 1e3)


def kernel_source_hash():
    h = hashlib.sha256()
    for f in ("toc_device.hip", "toc_host.cpp", "toc_internal.h"):
        h.update(open(os.path.join(HERE, "paper_1702_06943_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(op, cfg):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it was
    taken on the current kernel sources; else None."""
    path = os.path.join(HERE, "profiles", f"toc_kernels_{cfg}_hbm_traffic.txt")
    if not os.path.exists(path):
        return None
    src = kernel_source_hash()
    for line in open(path):
        parts = line.split()
        if len(parts) >= 4 and parts[0] == "traffic" and parts[1] == op and parts[2] == src:
            return float(parts[3])
    return None


# ---------------------------------------------------------------------------
def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default="c3", help="workload c1..c5 (default c3)")
    ap.add_argument("--batches", type=int, default=0,
                    help="mini-batches (default: the workload's full count)")
    ap.add_argument("--k", type=int, default=0, help="width of W and G (default: workload's)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="CPU time budget of the oracle baseline (0 = skip)")
    ap.add_argument("--workers", type=int, default=0)
    ap.add_argument("--no-extras", action="store_true",
                    help="skip timing the element-wise operations, the C' build and the "
                         "MGD epoch after the step")
    ap.add_argument("--nn-steps", type=int, default=2000,
                    help="neural-network MGD steps to time (0: skip)")
    ap.add_argument("--encode-batches", type=int, default=4000,
                    help="batches for the device encoder's measurement (0: skip)")
    ap.add_argument("--cprime-batches", type=int, default=4000,
                    help="batches whose physical encoding is turned into C' on the GPU "
                         "after the step (0 = skip)")
    ap.add_argument("--k1-extras", default="c5,c2",
                    help="k = 1 workloads timed after the step at full size (comma list; "
                         "empty: none)")
    ap.add_argument("--ingest", type=int, default=1,
                    help="1: after the step, build the whole image on the device from its "
                         "physical bytes and compare it with the host-built one")
    ap.add_argument("--copy-calib-mib", type=int, default=0,
                    help="after timing, copy this many MiB device-to-device three times "
                         "(reference dispatches for HBM byte counters)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on exactly one GPU: there is no multi-GPU path (batches are "
              "independent, so each GPU would take a contiguous range of them with W "
              "replicated).", file=sys.stderr)
        sys.exit(2)

    from workloads import CONFIGS
    from workloads.parallel import default_workers, make_pool
    cfg = args.config
    spec = CONFIGS[cfg]
    nb = args.batches or spec["n_batches"]
    k = args.k or spec["k"]
    workers = args.workers or default_workers()

    # everything that forks happens before the GPU is touched
    pool = make_pool(workers)
    cpu = cpu1 = None
    if args.cpu_seconds > 0:
        log(f"oracle CPU baseline on {workers} processes ...")
        cpu = cpu_baseline(pool, workers, cfg, nb, k, args.cpu_seconds)
        log(f"oracle: {cpu['value']:.3e} nnz/s ({cpu['sample']})")
        cpu1 = cpu_baseline_single(cfg, nb, k, args.cpu_seconds / 3)
        log(f"oracle on one core: {cpu1['value']:.3e} nnz/s ({cpu1['sample']})")
    w = encode_workload(cfg, nb, pool,
                        keep_batches=0 if args.no_extras else args.encode_batches)
    k1 = []
    if not args.no_extras:
        for c in [x for x in args.k1_extras.split(",") if x and x != cfg]:
            log(f"k = 1 extra {c}: generate and encode")
            k1.append(encode_workload(c, CONFIGS[c]["n_batches"], pool))
    pool.close()
    pool.join()

    import torch
    import paper_1702_06943_amd as T
    upload_workload(w, k)
    sample = None if args.no_extras else pack_sample(w, args.cprime_batches)
    packed = pack_all(w) if args.ingest and not args.no_extras else None
    ablation = variant_sizes(_host_map(T.toc_enc_info_get, w.encs), w.n_cols)
    encode_dev = None if args.no_extras else time_encode_device(w, torch.cuda.current_stream())
    w.encs = w.kept = None

    stream = torch.cuda.current_stream()
    log(f"warmup {args.warmup} steps, then {args.steps} timed")
    names = ("right", "left", "decode")
    op_ms, step_ms, t_wall = time_ops(w, args.steps, args.warmup, stream, names)
    log(f"step {step_ms:.3f} ms ({', '.join(f'{o} {op_ms[o]:.3f}' for o in names)}); "
        f"wall {t_wall / args.steps * 1e3:.3f} ms/step")
    if args.copy_calib_mib > 0:
        n = args.copy_calib_mib * (1 << 20) // 4
        src = torch.ones(n, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copy calibration: 3 copies of {n * 4} bytes")
        del src, dst

    copy_bw = measured_copy_bandwidth(stream)
    info = w.info
    extras = None if args.no_extras else time_elementwise(w, stream)
    cprime = time_cprime(sample, stream) if sample else None
    mgd = None if args.no_extras else time_mgd(w, stream)
    nn = None if args.no_extras else time_mlp(w, stream, args.nn_steps)
    k1res = time_k1_workloads(k1, args.steps, args.warmup, stream) if k1 else None
    ingest = time_ingest(w, packed) if packed else None
    packed = None
    nnz = info["nnz"]
    canon = info["canon_bytes"]
    m = info["n_cols"]
    # algorithmic bytes and flops per op (whole workload = one launch of each op)
    dense, flops = op_bytes_flops(info, k)
    ops = op_report(info, k, op_ms, copy_bw)
    dom = max(("right", "left", "decode"), key=lambda o: op_ms[o])
    t_dom = op_ms[dom] / 1e3
    bytes_dom = canon + dense[dom]
    intensity = flops[dom] / bytes_dom
    if intensity > FP32_PEAK / HBM_PEAK:
        roof = {"bound": "alu", "achieved": flops[dom] / t_dom / 1e12,
                "peak": FP32_PEAK / 1e12, "unit": "TFLOP/s"}
        roof["frac"] = roof["achieved"] / roof["peak"]
        # the same against one FMA per lane and clock (no packed FP32)
        roof["peak_nonpacked"] = FP32_NONPACKED_PEAK / 1e12
        roof["frac_nonpacked"] = roof["achieved"] / roof["peak_nonpacked"]
    else:
        roof = {"bound": "hbm", "achieved": bytes_dom / t_dom / 1e9,
                "peak": HBM_PEAK / 1e9, "unit": "GB/s"}
        roof["frac"] = roof["achieved"] / roof["peak"]
    full_size = nb == spec["n_batches"] and k == spec["k"]
    roof["traffic"] = measured_traffic(dom, cfg) if full_size else None
    roof["kernel"] = dom

    line = {
        "metric": METRIC,
        "value": nnz / (step_ms / 1e3),
        "unit": "nnz/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": step_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": f"{cfg}: {spec['name']}, {nb} mini-batches x {spec['rows']} rows x "
                        f"{m} columns, W {m}x{k}, G {spec['rows']}x{k} per batch",
            "batches": nb, "rows_per_batch": spec["rows"], "cols": m, "k": k,
            "nnz": nnz, "codes": info["n_codes"], "live_codes": info["n_stored"],
            "canon_bytes": canon, "image_bytes": info["image_bytes"],
            "step": "right_mul + left_mul + decode_csr over all batches",
        },
        "hbm_frac_compressed": {op: ops[op]["hbm_frac_compressed"] for op in names},
        "ops": ops,
        "roofline": roof,
        "elementwise": extras,
        "cprime_build": cprime,
        "device_ingest": ingest,
        "mgd_epoch": mgd,
        "nn_steps": nn,
        "k1_workloads": k1res,
        "encode_device": encode_dev,
        "ablation_sizes": ablation,
        "cpu_baseline": cpu,
        "cpu_baseline_single_thread": cpu1,
        "measured_copy_GBps": copy_bw / 1e9,
        "host": {"encode_s": round(w.encode_s, 2), "upload_s": round(w.upload_s, 2),
                 "cpu": host_cpu()},
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
