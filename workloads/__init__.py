"""Seeded synthetic workloads for the MoE-layer forward pass.

This package only draws random numbers and lays them out; it holds none of the
layer's arithmetic. Both the GPU path's tests and the CPU oracle's tests take
their inputs from here, so neither side generates data for the other.
"""

from .configs import CONFIGS, LayerConfig, get_config  # noqa: F401
from .generate import (  # noqa: F401
    LayerInputs,
    bf16_bits_to_f32,
    f32_to_bf16_bits,
    make_inputs,
    pad_last_dim,
)
