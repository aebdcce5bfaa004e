"""Seeded synthetic decode workloads for the weightless-attention-node path.

This package only draws and lays out inputs: query vectors, paged K/V pools,
token-range routes and page tables, and the per-step new K/V tokens.  It holds
none of the attention arithmetic.  Both the HIP path (through the Python
binding) and the CPU oracle consume what it produces; it imports neither.
"""
from .synth import (  # noqa: F401
    WORKLOADS,
    Workload,
    Instance,
    make_instance,
    workload,
    f32_to_bf16_bits,
    bf16_bits_to_f32,
    e4m3_encode,
)
