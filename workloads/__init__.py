"""Seeded synthetic inputs for the additively-quantized (AQ) layer forward and codebook gradient.

This package only draws random numbers and does shape bookkeeping; it holds
none of the AQ arithmetic (no decode, no matmul).  Both the CPU oracle tests
and the GPU path consume the arrays it produces, so neither side ever takes an
input from the other.
"""
from .layers import (  # noqa: F401
    ConvGeom,
    LayerSpec,
    generate,
    generate_grad_inputs,
    CONFIGS,
    config_spec,
    config_inputs,
    sweep_layers,
    sweep_spec,
    sweep_io_elems,
    chain_sources,
    branch_inputs,
    chain_codebook_std,
    lut_regime_specs,
    SEED_BASE,
)
