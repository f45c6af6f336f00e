"""Seeded synthetic attention inputs shared by the oracle, the GPU tests and the bench.

This package only draws and rounds numbers: it holds none of the attention method's
arithmetic, so both sides of every parity check consume bit-identical bf16 inputs
without sharing any code that computes attention.
"""

from .video_qkv import (
    WORKLOADS,
    Workload,
    bf16_bits,
    position_features,
    make_random_qkv,
    make_video_qkv,
    workload_inputs,
)
from .half_flip import half_flip_inputs
from .margin_band import margin_band_inputs
from .vote_patterns import expected_skip, vote_pattern_inputs

__all__ = [
    "WORKLOADS",
    "Workload",
    "bf16_bits",
    "position_features",
    "make_random_qkv",
    "make_video_qkv",
    "workload_inputs",
    "vote_pattern_inputs",
    "margin_band_inputs",
    "half_flip_inputs",
    "expected_skip",
]
