"""Seeded synthetic inputs for the cached attention layer.

This package only draws random tensors and rounds them to the storage dtype.
It holds none of the caching method's arithmetic (no similarity, no
selection, no attention), so both the CPU oracle's tests and the HIP path's
tests and benchmark may use it as their common source of inputs.
"""
from .workloads import (  # noqa: F401
    WORKLOADS,
    Workload,
    bf16_bits,
    bf16_bits_to_f32,
    ffn_weights,
    layered_tables,
    make_workload,
    small_workload,
)
