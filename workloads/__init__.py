"""Seeded synthetic inputs shared by the GPU path's tests/benchmark and the CPU oracle."""
from .synth import (  # noqa: F401
    sub_row_pairing,
    BLOCK, C4_SWEEP, HEAD_DIM, WORKLOADS, Workload, bf16_bits_to_f32, generate,
    random_bf16, random_score_rows, small, to_bf16_bits,
)
