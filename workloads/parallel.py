"""Process-parallel generation of a workload's mini-batches, in order, in chunks.

Use before any GPU initialisation in the calling process (the pool forks).
"""

from __future__ import annotations

import multiprocessing as mp
import os

from .gen import CONFIGS, config_batches


def default_workers():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _make(args):
    cfg, first, count = args
    return config_batches(cfg, first, count)


def iter_chunks(cfg, n_batches=None, first=0, chunk=200, pool=None):
    """Yields Batches objects of consecutive chunks of the workload, in order."""
    n_batches = CONFIGS[cfg]["n_batches"] if n_batches is None else n_batches
    jobs = [(cfg, b, min(chunk, first + n_batches - b))
            for b in range(first, first + n_batches, chunk)]
    if pool is None:
        for j in jobs:
            yield _make(j)
        return
    yield from pool.imap(_make, jobs)


def make_pool(workers=None):
    return mp.get_context("fork").Pool(workers or default_workers())
