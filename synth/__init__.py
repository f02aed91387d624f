"""Seeded synthetic inputs for the RBS sparse-prefill path.

This package only draws random numbers and lays them out; it holds none of the
method's arithmetic (no block statistics, scores, selection or attention).  The
oracle, the tests and the benchmark all read the same bf16 arrays from here.
"""

from .bf16 import bf16_bits_from_f32, f32_from_bf16_bits, f64_from_bf16_bits
from .workloads import (
    Workload,
    WORKLOADS,
    workload,
    make_inputs,
    layer_schedule,
    batch_workloads,
    make_batch_inputs,
)

__all__ = [
    "bf16_bits_from_f32",
    "f32_from_bf16_bits",
    "f64_from_bf16_bits",
    "Workload",
    "WORKLOADS",
    "workload",
    "make_inputs",
    "layer_schedule",
    "batch_workloads",
    "make_batch_inputs",
]
