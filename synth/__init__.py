"""Seeded synthetic workloads for the ARCHead packed LM-head forward.

This package draws inputs only: packed heads (INT4 code bytes, fp16 scales,
INT8 factors), bf16 hidden states and target ids.  It holds none of the
method's arithmetic (no unpacking, no dequantisation, no logits), so both the
HIP path and the CPU oracle can consume the same bytes without sharing code.
"""
from .gen import (  # noqa: F401
    CONFIGS,
    HeadArrays,
    make_head,
    make_x,
    make_targets,
    make_workload,
    f64_to_bf16_bits,
)
