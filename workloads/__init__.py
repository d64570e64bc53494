"""Seeded synthetic workloads for the COUNTDOWN sparse Gated-MLP FFN.

This package only draws random numbers and lays them out; it holds none of
the method's arithmetic. Both the CPU oracle (through the tests) and the HIP
path (through the tests and the bench) receive the same arrays from here.
"""
from .synth import (  # noqa: F401
    ROOT_SEED,
    WORKLOADS,
    Workload,
    bf16_round,
    bf16_to_f32,
    make_layer,
    make_low_rank,
    make_predictor,
    make_ternary,
    make_tokens,
    outlier_channels,
    stream,
)
