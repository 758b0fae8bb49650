"""Seeded synthetic inputs for Sparse Feature Attention workloads.

This module only *draws* inputs.  It holds none of the method's arithmetic:
no Top-k selection, no scores, no softmax.  Both the CPU oracle (in tests)
and the GPU path consume what it produces, so a parity test compares the
two on identical bytes.

Every tensor slice is drawn from its own generator, seeded by a stable hash
of (workload seed, tensor name, batch, head).  A single (b, h) slice can
therefore be regenerated on its own -- this is how tests and the benchmark
hand the oracle the exact inputs of a sampled slice of a large workload.

The values of a slice depend on the device it is drawn on (torch's CPU and
GPU generators differ), so producer and consumer of one comparison must use
the same device for generation.
"""
from .gen import (  # noqa: F401
    slice_seed,
    normal,
    to_bf16,
    dense_qkv,
    zipf_feature_perm,
    zipf_codes,
    dense_from_codes,
    tie_rows,
    random_csr,
)
from .configs import WORKLOADS, Workload, workload  # noqa: F401
