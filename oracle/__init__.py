"""CPU oracle for the additively-quantized (AQ) layer forward and codebook gradient.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package.  The GPU library never
calls it and shares no code with it: it is the plain, slow, fp64 statement of
what the layer computes, used to judge the GPU kernels.
"""
from .aq_oracle import (  # noqa: F401
    to_f64,
    dequantize,
    activations_f64,
    im2col,
    linear_forward,
    conv_forward,
    forward,
    forward_sampled,
    decode_emulate,
    f32_to_bf16_bits,
    bf16_bits_to_f32,
    rel_err_inf,
    rel_err_rms,
    rel_err_elem,
    abs_inputs,
    rounding_bound,
    dense_conv_flops,
    lut_conv_flops,
    lut_breakpoint_cout,
    weight_grad_linear,
    weight_grad_conv,
    codebook_grad_from_weight_grad,
    codebook_grad,
    codebook_grad_entries,
)
