"""GPU parity of the codebook gradient (through the C ABI) against the fp64 oracle.

X and dY are stored in fp16 or bf16 and widen exactly, products of two such
values are exact in fp32, and every sum runs in fp32: over tokens for the
weight gradient (N up to 8192), then over the (row, group) pairs that share a
codebook entry.  The relative error of an fp32 sum of n random-sign terms
grows like 2^-24 * sqrt(n), about 5e-6 for n = 8192, so the bar is an
infinity-norm relative error (max |dC - dC*| / max |dC*|) of 2e-5.
Summation orders are fixed, so repeated calls must agree bit for bit.
"""
import dataclasses
import os
import sys

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from workloads import ConvGeom, LayerSpec, generate, generate_grad_inputs

pytestmark = pytest.mark.gpu

TOL = 2e-5


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need an MI355X; none is visible")
    import paper_2506_05960_amd as P
    P.load_library()
    yield


def _dev(a, dt):
    a = np.ascontiguousarray(a)
    if dt == "bf16":
        return torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(a).cuda()


def _grad(spec, inp, gi, dt, splits=None, layer=None, opts=None):
    import paper_2506_05960_amd as P
    own = layer is None
    if own:
        layer = P.AQLayer(spec, inp)
    for k, v in (opts or {}).items():
        layer.set_option(k, v)
    if splits is not None:
        layer.set_option("grad_splits", splits)
    x, dy = _dev(gi["x"], dt), _dev(gi["dy"], dt)
    out = layer.codebook_grad(x, dy)
    torch.cuda.synchronize()
    if splits is not None:
        layer.set_option("grad_splits", 0)
    res = out.cpu().numpy().astype(np.float64)
    if own:
        layer.close()
    return res


def _ref(spec, inp, gi, dt):
    return O.codebook_grad(spec, {"codes": inp["codes"], "scales": inp["scales"], "x": gi["x"]}, gi["dy"],
                           x_dtype=dt, dy_dtype=dt)


def _lin(name, C_out, K, g, M, B, n):
    return LayerSpec(name=name, C_out=C_out, K=K, g=g, M=M, B=B, n=n)


def _conv(name, cin, C_out, H, W_, k, g, M, B, n):
    geom = ConvGeom(cin=cin, kh=k, kw=k, stride=1, pad=k // 2, H=H, W=W_)
    return LayerSpec(name=name, C_out=C_out, K=geom.K, g=g, M=M, B=B, n=n, conv=geom)


CASES = [
    # one tile, a ragged token tail (N not a multiple of 64)
    (_lin("lin_small", 64, 64, 8, 2, 8, 100), "f16"),
    # several tiles in both directions, partial tiles, ragged tokens
    (_lin("lin_tiles", 200, 328, 8, 4, 8, 517), "f16"),
    (_lin("lin_bf16", 136, 256, 8, 2, 6, 300), "bf16"),
    (_lin("lin_g9", 72, 144, 9, 2, 5, 130), "f16"),
    (_lin("lin_m1_b12", 96, 192, 8, 1, 12, 260), "f16"),
    (_lin("lin_b16", 64, 128, 8, 1, 16, 70), "f16"),
    (_lin("lin_g16_m3", 48, 256, 16, 3, 4, 90), "f16"),
    (_lin("lin_one_token", 64, 64, 8, 2, 8, 1), "f16"),
    # 3x3 convolutions: several channel tiles, rows with halo, odd image counts
    (_conv("conv3_small", 16, 32, 8, 8, 3, 8, 2, 8, 2), "f16"),
    (_conv("conv3_tiles", 40, 136, 6, 16, 3, 8, 2, 8, 3), "f16"),
    (_conv("conv3_g9_kaq", 24, 64, 8, 8, 3, 9, 2, 8, 2), "f16"),
    (_conv("conv3_bf16", 16, 80, 8, 24, 3, 8, 1, 10, 1), "bf16"),
    (_conv("conv3_b16", 32, 64, 4, 8, 3, 8, 1, 16, 2), "f16"),
    # 64-token chunks that are whole output rows (the direct-to-LDS kernel)
    (_conv("conv3_w16", 24, 72, 8, 16, 3, 8, 2, 8, 2), "f16"),
    (_conv("conv3_w32_bf16", 16, 136, 4, 32, 3, 8, 2, 7, 3), "bf16"),
    (_conv("conv3_w64", 8, 40, 3, 64, 3, 8, 1, 9, 1), "f16"),
    # 1x1 convolutions
    (_conv("conv1", 64, 96, 8, 8, 1, 8, 2, 8, 3), "f16"),
    (_conv("conv1_g16", 128, 40, 4, 16, 1, 16, 4, 6, 2), "bf16"),
]


@pytest.mark.parametrize("spec,dt", CASES, ids=[c[0].name + "_" + c[1] for c in CASES])
def test_codebook_grad_matches_oracle(spec, dt):
    _say(f"[grad] {spec.name} {dt}")
    inp = generate(spec, 31)
    gi = generate_grad_inputs(spec, 32, dt)
    got = _grad(spec, inp, gi, dt)
    ref = _ref(spec, inp, gi, dt)
    assert got.shape == ref.shape
    err = O.rel_err_inf(got, ref)
    assert err <= TOL, err


SPLIT_CASES = [c for c in CASES if c[0].name in ("lin_tiles", "conv3_tiles", "conv3_w16", "conv1")]


@pytest.mark.parametrize("spec,dt", SPLIT_CASES, ids=[c[0].name for c in SPLIT_CASES])
def test_token_splits_agree(spec, dt):
    """One split and the planner's split count give the same gradient within the bar."""
    _say(f"[grad splits] {spec.name}")
    inp = generate(spec, 33)
    gi = generate_grad_inputs(spec, 34, dt)
    a = _grad(spec, inp, gi, dt, splits=1)
    b = _grad(spec, inp, gi, dt)
    ref = _ref(spec, inp, gi, dt)
    assert O.rel_err_inf(a, ref) <= TOL
    assert O.rel_err_inf(b, ref) <= TOL


DMA_CASES = [c for c in CASES if c[0].name in ("lin_small", "lin_tiles", "lin_bf16", "lin_one_token", "conv3_small",
                                                "conv3_g9_kaq", "conv3_w16", "conv1", "conv1_g16")]


@pytest.mark.parametrize("spec,dt", DMA_CASES, ids=[c[0].name for c in DMA_CASES])
def test_direct_to_lds_and_register_staged_kernels_agree(spec, dt):
    """Layers eligible for the direct-to-LDS kernels, also run through the register-staged ones."""
    _say(f"[grad dma vs regs] {spec.name}")
    inp = generate(spec, 46)
    gi = generate_grad_inputs(spec, 47, dt)
    ref = _ref(spec, inp, gi, dt)
    for tile in ("64x64", "128x64"):
        a = _grad(spec, inp, gi, dt, opts={"grad_tile": tile})
        assert O.rel_err_inf(a, ref) <= TOL, tile
    b = _grad(spec, inp, gi, dt, opts={"grad_regs": 1})
    assert O.rel_err_inf(b, ref) <= TOL


def test_repeated_calls_are_bitwise_identical():
    import paper_2506_05960_amd as P
    spec, dt = CASES[1]
    _say("[grad repeat]")
    inp = generate(spec, 35)
    gi = generate_grad_inputs(spec, 36, dt)
    layer = P.AQLayer(spec, inp)
    a = _grad(spec, inp, gi, dt, layer=layer)
    b = _grad(spec, inp, gi, dt, layer=layer)
    layer.close()
    assert np.array_equal(a, b)


def test_fewer_tokens_than_created_for():
    """A layer sized for many tokens takes a smaller call (fewer chunks than splits)."""
    import paper_2506_05960_amd as P
    spec, dt = CASES[1]
    big = dataclasses.replace(spec, n=4096)
    inp = generate(big, 37)
    layer = P.AQLayer(big, inp)
    small = dataclasses.replace(spec, n=65)
    gi = generate_grad_inputs(small, 38, dt)
    _say("[grad small call]")
    got = _grad(small, inp, gi, dt, layer=layer)
    layer.close()
    assert O.rel_err_inf(got, _ref(small, inp, gi, dt)) <= TOL


def test_gradient_of_codes_never_used_is_zero():
    spec, dt = CASES[0]
    inp = generate(spec, 39)
    inp["codes"] = (inp["codes"] % 16).astype(inp["codes"].dtype)
    gi = generate_grad_inputs(spec, 40, dt)
    _say("[grad unused codes]")
    got = _grad(spec, inp, gi, dt)
    assert np.all(got[:, 16:, :] == 0.0)
    assert O.rel_err_inf(got, _ref(spec, inp, gi, dt)) <= TOL


def test_unsupported_layers_are_rejected():
    import paper_2506_05960_amd as P
    stride2 = LayerSpec(name="s2", C_out=32, K=16 * 9, g=8, M=2, B=8, n=1,
                        conv=ConvGeom(cin=16, kh=3, kw=3, stride=2, pad=1, H=8, W=8))
    odd = _lin("odd", 36, 64, 8, 2, 8, 8)
    for spec in (stride2, odd):
        inp = generate(spec, 41)
        layer = P.AQLayer(spec, inp)
        gi = generate_grad_inputs(spec, 42, "f16")
        with pytest.raises(P.AQError, match="AQ_ERR_UNSUPPORTED"):
            layer.codebook_grad(_dev(gi["x"], "f16"), _dev(gi["dy"], "f16"))
        layer.close()


FULL = [("qkv16", "f16"), ("conv64", "f16"), ("conv8", "f16")]


@pytest.mark.parametrize("cfg,dt", FULL, ids=[c[0] for c in FULL])
def test_full_size_sampled_entries(cfg, dt):
    """Full workload shapes (fp16 inputs), checked on sampled codebook entries the oracle evaluates one by one."""
    spec = W.config_spec(cfg)
    if spec.x_dtype != dt:
        spec = dataclasses.replace(spec, x_dtype=dt)
    _say(f"[grad full] {cfg}")
    inp = W.generate(spec, 43)
    gi = generate_grad_inputs(spec, 44, dt)
    got = _grad(spec, inp, gi, dt)
    rng = np.random.default_rng(45)
    nk = 1 << spec.B
    entries = [(int(rng.integers(spec.M)), int(rng.integers(nk))) for _ in range(12)]
    # the most and least used entries of codebook 0 as well
    counts = np.bincount(inp["codes"][:, :, 0].reshape(-1).astype(np.int64), minlength=nk)
    entries += [(0, int(np.argmax(counts))), (0, int(np.argmin(counts)))]
    ref = O.codebook_grad_entries(spec, {"codes": inp["codes"], "scales": inp["scales"], "x": gi["x"]}, gi["dy"],
                                  entries, x_dtype=dt, dy_dtype=dt)
    sel = np.stack([got[m, k] for m, k in entries])
    den = np.max(np.abs(ref))
    assert den > 0
    assert np.max(np.abs(sel - ref)) / den <= TOL
