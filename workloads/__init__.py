"""Seeded synthetic workloads for the ReTrace round: shape presets and input generators.

This package holds configuration and random-input generation only.  It contains
none of the method's arithmetic, so both the CPU oracle and the GPU harness may
import it without sharing any computation.
"""
from .configs import Workload, ModelShape, PRESETS, get, cond_layer_ids
from .generate import (weight_specs, make_weights, make_prompts, bf16_bits_to_f32,
                       f32_to_bf16_bits)

__all__ = ["Workload", "ModelShape", "PRESETS", "get", "cond_layer_ids", "weight_specs",
           "make_weights", "make_prompts", "bf16_bits_to_f32", "f32_to_bf16_bits"]
