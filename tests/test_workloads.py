"""Seeded input generators: shapes, dtypes, ranges, determinism, layer list."""
import json
import os

import numpy as np
import pytest

import workloads as W
from workloads.layers import unet_attention_macs, unet_unquantized_conv_macs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.mark.parametrize("name", ["tiny", "conv64", "qkv16", "conv8"])
def test_config_shapes_and_dtypes(name):
    spec = W.config_spec(name)
    inp = W.config_inputs(name)
    M, B, g = spec.M, spec.B, spec.g
    assert inp["codebooks"].shape == (M, 1 << B, g)
    assert inp["codes"].shape == (spec.C_out, spec.K // g, M)
    assert inp["codes"].dtype == (np.uint8 if B <= 8 else np.uint16)
    assert int(inp["codes"].max()) < (1 << B)
    assert inp["scales"].dtype == np.float32 and inp["scales"].shape == (spec.C_out,)
    assert 0.5 <= inp["scales"].min() and inp["scales"].max() <= 1.5
    if spec.conv is None:
        assert inp["x"].shape == (spec.n, spec.K)
    else:
        c = spec.conv
        assert inp["x"].shape == (spec.n, c.cin, c.H, c.W)
    if spec.x_dtype == "i8":
        assert inp["x"].dtype == np.int8 and inp["x"].min() >= -127
        assert inp["x_scales"].shape == (spec.tokens,)
    else:
        assert inp["x_scales"] is None


def test_generation_is_deterministic():
    a = W.config_inputs("tiny")
    b = W.config_inputs("tiny")
    for k in ("codebooks", "codes", "scales", "x"):
        assert np.array_equal(a[k], b[k])


def test_config_sizes():
    assert W.config_spec("conv64").tokens == 8192 and W.config_spec("conv64").K == 1728
    assert W.config_spec("qkv16").tokens == 8192
    assert W.config_spec("conv8").tokens == 4096 and W.config_spec("conv8").K == 8640
    assert W.config_spec("conv64").dense_flops == 2 * 8192 * 1728 * 192


def test_bits_per_weight_golden():
    gold = json.load(open(os.path.join(GOLDEN, "bits_per_weight.json")))
    for c in gold["cases"]:
        assert c["M"] * c["n"] / c["g"] == pytest.approx(c["bits"])
    for name, bits in (("tiny", 2), ("conv64", 2), ("qkv16", 4), ("conv8", 2)):
        s = W.config_spec(name)
        assert s.M * s.B / s.g == bits


def test_sweep_layer_list_checksums():
    strict, full = W.sweep_layers(False), W.sweep_layers(True)
    assert len(strict) == 97 and len(full) == 209
    assert len({(l.kind, l.cin, l.cout, l.res, l.stride) for l in strict}) == 42
    assert sum(l.macs(8) for l in strict) * 2 / 1e9 == pytest.approx(1202.71, abs=0.01)
    assert sum(l.macs(8) for l in full) * 2 / 1e9 == pytest.approx(1595.47, abs=0.01)


def test_sweep_matches_table3_fp_total():
    """Soft checksum: the layer list plus attention matmuls and conv_in/out vs Table 3."""
    gold = json.load(open(os.path.join(GOLDEN, "table3_fp_gmac.json")))
    b = gold["batch"]
    tot = sum(l.macs(b) for l in W.sweep_layers(True)) + unet_attention_macs(b) + unet_unquantized_conv_macs(b)
    assert abs(tot / 1e9 - gold["fp_gmac"]) / gold["fp_gmac"] < 0.005


def test_sweep_specs_are_valid():
    for l in W.sweep_layers(True):
        for M in (2, 4):
            s = W.sweep_spec(l, M)
            assert s.K % s.g == 0
            if s.conv is not None:
                assert s.conv.OH == l.res // l.stride


def test_branch_inputs_are_the_residual_skips():
    """Every residual skip convolution (and nothing else) shares the input of its block's first 3x3 convolution,
    which comes before it and has the same input shape."""
    for full in (False, True):
        layers = W.sweep_layers(full)
        br = W.branch_inputs(layers)
        assert [i for i, j in enumerate(br) if j is not None] == [i for i, l in enumerate(layers) if l.role == "res_skip"]
        assert sum(j is not None for j in br) == 15
        for i, j in enumerate(br):
            if j is None:
                continue
            a, b = layers[i], layers[j]
            assert j < i and b.name == a.name.rsplit(".", 1)[0] + ".conv1" and b.kind == "conv3x3"
            assert (a.cin, a.res, a.stride) == (b.cin, b.res, b.stride)
            assert W.sweep_io_elems(a, 8)[0] == W.sweep_io_elems(b, 8)[0]
