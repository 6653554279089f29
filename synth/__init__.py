"""Seeded synthetic inputs shared by the oracle tests, the GPU tests and the benchmark.

This package only draws and shapes random inputs (Gaussian Q/K/V, rotary position
encoding, planted structure, bf16 rounding).  It holds none of the attention, probe,
index, coverage or routing arithmetic.
"""
from .gen import (CONFIGS, LayerSpec, layer_spec, make_layer, bf16_round, bf16_bits,
                  bits_to_f32)

__all__ = ["CONFIGS", "LayerSpec", "layer_spec", "make_layer", "bf16_round", "bf16_bits",
           "bits_to_f32"]
