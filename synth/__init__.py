"""Seeded synthetic workloads for the packed four-direction MDLSTM layer.

This package only draws random numbers: example sizes, pixel/feature values,
weights and upstream gradients. It holds none of the method's arithmetic, so
both the CPU oracle (``oracle/``) and the HIP path's tests and benchmark can
draw identical inputs from it without sharing any computation.
"""
from .configs import (  # noqa: F401
    Workload,
    StackWorkload,
    workload,
    stack_workload,
    round_to_bf16,
    padded_fraction,
)
