"""Seeded synthetic inputs for the mixed-adapter LoRA layer.

This package only draws and encodes inputs (structure, values, dtype encoding).
It holds none of the layer's arithmetic, so both the float64 oracle and the HIP
path can be fed from it without sharing any computation.
"""
from .encode import (bf16_bits_from_f64, f64_from_bf16_bits, f32_from_f64,
                     encode, decode)
from .configs import (Case, CONFIG_NAMES, base_weight, make_config, random_case,
                      segments_to_idx)

__all__ = ["bf16_bits_from_f64", "f64_from_bf16_bits", "f32_from_f64", "encode",
           "decode", "Case", "CONFIG_NAMES", "base_weight", "make_config", "random_case",
           "segments_to_idx"]
