"""Seeded synthetic mini-batch generators shared by the tests and the benchmark.

Holds no part of the compression or of the products: it only draws inputs
(CSR mini-batches, W and G) with the shapes and value structure of the paper's
workloads.  Both the oracle and the HIP path are fed from here.
"""

from .gen import (  # noqa: F401
    CONFIGS,
    SEED,
    Batches,
    config_batches,
    config_W,
    config_G,
    tiny_batch,
    dense_normal,
    dense_normal_device,
)
