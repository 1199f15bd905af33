"""Seeded synthetic workloads for compressed-KV decode attention.

This package is shared harness code: it draws the random inputs (activations,
queries, factor matrices, pre-filled latents, ragged lengths, page tables) for
both the GPU path and the CPU oracle.  It holds none of the method's
arithmetic -- no projection, rounding of results, softmax or layout
computation -- only the construction of inputs and their shapes.
"""

from .configs import (  # noqa: F401
    PAGE_TOKENS,
    WORKLOAD_NAMES,
    Workload,
    make_workload,
)
from .inputs import Inputs, make_inputs, bf16_bits_from_f32, f32_from_bf16_bits  # noqa: F401
