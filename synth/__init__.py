"""Seeded synthetic inputs for the ACE MoE layer.

This package only draws random numbers and rounds them to the storage dtype.
It holds none of the method's arithmetic, so both the CPU oracle's tests and
the GPU path's tests and benchmark can take their inputs from it without the
two sides sharing any computation.
"""
from .configs import CONFIGS, STACK_LAYERS, LayerConfig, config
from .gen import (
    bf16_bits_to_f32,
    decode_inputs,
    f32_to_bf16_bits,
    make_layer,
    rng_for,
)

__all__ = [
    "CONFIGS",
    "STACK_LAYERS",
    "LayerConfig",
    "config",
    "bf16_bits_to_f32",
    "decode_inputs",
    "f32_to_bf16_bits",
    "make_layer",
    "rng_for",
]
