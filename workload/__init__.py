"""Seeded synthetic inputs for the EAT MoE layer.

This module only draws random numbers and packs them into arrays (fp32, or
bf16 bit patterns as uint16).  It holds none of the routing or expert
arithmetic, so both the CPU oracle's tests and the GPU path can take their
inputs from it without sharing any of the method's code.
"""
from .gmm import (  # noqa: F401
    LayerShape,
    SHAPES,
    bf16_bits,
    make_layer_weights,
    make_mixing,
    make_expert_scale,
    make_vocab_head,
    make_targets,
    HiddenStream,
    make_prefill,
    make_trend,
    make_accounts,
)
