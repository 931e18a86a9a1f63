"""Seeded synthetic inputs for the future-attention target.

This package is shared by the fp64 oracle's tests and by the GPU path's tests and
benchmark. It holds only input generation: random draws, RMS normalisation, rotary
position embedding and rounding to bfloat16. None of the target's arithmetic
(logits, log-normalisers, probabilities, future mass) lives here.
"""
from .gen import (  # noqa: F401
    CONFIGS,
    Workload,
    bf16_round_bits,
    make,
    make_scores,
    make_slice,
    make_values,
    rmsnorm,
    rope,
)
