"""Seeded synthetic inputs shared by the CPU oracle's tests, the GPU parity
tests and the benchmark.

This package draws inputs only: hidden states, expert and router weights,
the block/mask layout of block-wise diffusion decoding and the confidence
histories.  It holds none of the method's arithmetic (no routing, budgeting,
ranking or expert computation), so that the oracle and the HIP path share
nothing but their inputs.
"""
from .workloads import (  # noqa: F401
    AllocParams,
    Workload,
    bf16_bits_from_f32,
    make_workload,
    make_fuzz_workload,
    WORKLOAD_NAMES,
)
from .trajectory import forward_confidence, generation_start  # noqa: F401
