"""Seeded synthetic workloads for the sparse sequence-parallel attention path.

This package only makes inputs: Q, K, V tensors of the shapes and value
distributions of the paper's video-DiT workloads, plus the geometry that goes
with them (block size, local query-block slice, keep count, global blocks).
It holds none of the method's arithmetic. Both the float64 oracle and the GPU
path consume exactly the bits it produces.
"""

from .synth import (  # noqa: F401
    CONFIGS,
    Workload,
    bf16_round_bits,
    get_workload,
    make_qkv,
    workload_names,
)
