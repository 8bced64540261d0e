"""Seeded synthetic inputs for the H-Scale hot path.

This module only draws random tensors; it holds none of the method's
arithmetic.  The oracle side (tests) and the HIP side (tests, smoke, bench)
both take their inputs from here.  The calibration data and model weights
the paper uses (FineWeb activations; Qwen3 and Llama-3 checkpoints) are not
available, so these distributions stand in for them with the shapes of 8B-
and 70B-class linear layers.
"""
from .workloads import (  # noqa: F401
    CONFIGS,
    Workload,
    make_activations,
    make_weight,
    harness_global_scale,
    bf16_bits_to_float,
)
