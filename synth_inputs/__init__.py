"""Seeded synthetic inputs for the HSA forward pass.

This module only draws random numbers and lays them out in the memory layout
the C ABI defines. It holds none of the method's arithmetic: no feature map,
no page index, no scores, no attention. Both the fp64 oracle (``oracle/``) and
the HIP path (through its Python binding) consume what it produces.
"""
from .configs import WORKLOADS, Workload, get_workload  # noqa: F401
from .gen import (  # noqa: F401
    Case,
    bf16_bits_to_f32,
    f32_to_bf16_bits,
    make_case,
    make_case_torch,
    make_projections,
    make_prompts,
    seed_int,
)
