"""Seeded synthetic inputs for the shared-KV-pool decode workloads.

This package only draws numbers and describes shapes: it holds none of the
attention arithmetic. Both the oracle side (tests, CPU baseline) and the HIP
side (tests, bench) take their inputs from here, so the two can be compared on
identical bytes.
"""
from .gen import (  # noqa: F401
    MODELS,
    ModelSpec,
    Workload,
    RequestSpec,
    make_workload,
    f32_to_bf16_bits,
    normal_bf16,
    algorithmic_bytes,
)
