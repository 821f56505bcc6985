"""Seeded synthetic KV-cache workloads.

This package only draws inputs: keys, values, queries and calibration samples with
LLM-like spectra.  It contains none of the compression method's arithmetic, so both
the CPU oracle and the GPU path may use it.
"""
from .gen import (  # noqa: F401
    CONFIGS,
    Workload,
    bf16_bits_to_f32,
    f32_to_bf16_bits,
    haar_orthogonal,
    layer_inputs,
    projection,
    workload,
)
