"""Seeded synthetic inputs for the LC-VQ linear layer.

This module is shared by the CPU oracle's tests, the GPU parity tests and the
benchmark.  It holds random draws and the fp32 -> bf16 storage cast only; none
of the layer's arithmetic (quantisation, decode, products, gradients) lives
here, so both sides of a parity check consume identical input bits without
sharing any of the method.
"""
from .inputs import (  # noqa: F401
    WORKLOADS,
    bf16_bits,
    bf16_bits_to_f32,
    draw_activations,
    draw_latent,
    draw_map,
    layer_inputs,
    rng,
)
