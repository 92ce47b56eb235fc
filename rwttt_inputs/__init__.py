"""Seeded synthetic inputs for the RW-TTT fast-weight READ/WRITE path.

This package is the only code shared by the GPU path's callers and the CPU
oracle.  It holds the workload table, the per-step role schedules and the
seeded tensor draws, and none of the method's arithmetic: no planning, no
apply, no update, no commit.
"""

from .workloads import (  # noqa: F401
    READ, WRITE, IDLE, WORKLOADS, Workload, workload, shape_class,
)
from .schedule import StepItem, build_trace  # noqa: F401
from .tensors import TensorSource, draw, f32_to_bf16_bits, bf16_bits_to_f32  # noqa: F401
