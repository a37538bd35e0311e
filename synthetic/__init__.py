"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark."""
from .workloads import (  # noqa: F401
    MID, P720, PYRAMID_GRIDS, SWEEP, SWEEP_DENSITIES, TINY, Workload,
    bf16_bits, bf16_to_f32, bf16_to_f64, generate, generate_head, head_densities,
    pyramid_scales,
)
