"""Seeded synthetic StepKV workloads.

This package only draws inputs (caches, observation windows, step spans and
the raw per-step signals). It contains none of the compression method's
arithmetic, so both the HIP path and the CPU oracle may consume what it
produces.
"""
from .workloads import (  # noqa: F401
    CONFIG_NAMES,
    SEEDS,
    StepSignals,
    Workload,
    bf16_bits_to_f32,
    f32_to_bf16_bits,
    make_workload,
)
