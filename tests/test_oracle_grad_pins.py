"""Pins of the fp64 codebook-gradient oracle against things other than itself.

The loss L(C) = <dY, Y(C)> is linear in the codebooks (eq. (4) is a sum of
codewords, and the layer is linear in its weights), so its gradient is fixed by
the forward alone: entry (m, k, t) equals L at the unit codebook E_mkt, and
<dC, V> = L(V) for every V.  The forward oracle is pinned by brute force in
the forward pin tests; the checks here reach the gradient through it, through
brute-force sums that never form dW, and through torch's autograd of an
independently written dequantization and of torch's own convolution.
"""
import math
import types

import numpy as np
import pytest
import torch

import oracle as O


def _spec(g, M, B, conv=None):
    return types.SimpleNamespace(g=g, M=M, B=B, codebook_dtype="f32", x_dtype="f32", conv=conv)


def _conv(kh, kw, stride, pad):
    return types.SimpleNamespace(kh=kh, kw=kw, stride=stride, pad=pad)


def _layer(rng, C_out, G, g, M, B):
    cb = rng.normal(0.0, 0.1, size=(M, 1 << B, g))
    codes = rng.integers(0, 1 << B, size=(C_out, G, M)).astype(np.uint8 if B <= 8 else np.uint16)
    s = rng.uniform(0.5, 1.5, size=C_out).astype(np.float32)
    return cb, codes, s


def _loss(spec, cb, codes, s, x, dy):
    """<dY, Y(C)> through the forward oracle."""
    y = O.forward(spec, {"codebooks": cb, "codes": codes, "scales": s, "x": x})
    return float(np.sum(y * dy))


@pytest.mark.parametrize("g,M,B", [(1, 1, 1), (2, 3, 2), (4, 2, 3), (9, 2, 2), (8, 1, 3)])
def test_every_entry_is_the_loss_at_its_unit_codebook(g, M, B):
    """dC[m, k, t] = L(E_mkt): the derivative of a linear function along a unit vector."""
    rng = np.random.default_rng(7 + g * 13 + M * 5 + B)
    C_out, G, N = 3, 3, 4
    cb, codes, s = _layer(rng, C_out, G, g, M, B)
    x = rng.normal(size=(N, G * g))
    dy = rng.normal(size=(N, C_out))
    spec = _spec(g, M, B)
    dC = O.codebook_grad(spec, {"codes": codes, "scales": s, "x": x}, dy)
    assert dC.shape == (M, 1 << B, g)
    for m in range(M):
        for k in range(1 << B):
            for t in range(g):
                E = np.zeros_like(cb)
                E[m, k, t] = 1.0
                assert abs(dC[m, k, t] - _loss(spec, E, codes, s, x, dy)) <= 1e-12 * (1 + abs(dC[m, k, t]))


def test_brute_force_sum_without_a_weight_gradient():
    """fsum over (n, i, j) of dY[n, i] * s_i * X[n, j*g + t] for every matching code."""
    rng = np.random.default_rng(11)
    g, M, B, C_out, G, N = 3, 2, 2, 4, 3, 5
    cb, codes, s = _layer(rng, C_out, G, g, M, B)
    x = rng.normal(size=(N, G * g))
    dy = rng.normal(size=(N, C_out))
    dC = O.codebook_grad(_spec(g, M, B), {"codes": codes, "scales": s, "x": x}, dy)
    for m in range(M):
        for k in range(1 << B):
            for t in range(g):
                terms = [float(dy[n, i]) * float(s[i]) * float(x[n, j * g + t])
                         for n in range(N) for i in range(C_out) for j in range(G) if int(codes[i, j, m]) == k]
                assert abs(dC[m, k, t] - math.fsum(terms)) <= 1e-13 * max(1.0, sum(abs(v) for v in terms))


def test_unused_codewords_get_zero_gradient():
    rng = np.random.default_rng(12)
    g, M, B, C_out, G, N = 4, 2, 4, 3, 2, 6
    cb, codes, s = _layer(rng, C_out, G, g, M, B)
    codes[..., 0] = codes[..., 0] % 4            # codebook 0 uses only entries 0..3
    x = rng.normal(size=(N, G * g))
    dy = rng.normal(size=(N, C_out))
    dC = O.codebook_grad(_spec(g, M, B), {"codes": codes, "scales": s, "x": x}, dy)
    assert np.all(dC[0, 4:] == 0.0)
    used = np.unique(codes[..., 1])
    assert np.all(np.any(dC[1, used] != 0.0, axis=-1))


@pytest.mark.parametrize("g,M,B", [(8, 2, 8), (8, 4, 8), (9, 2, 4), (8, 1, 16), (16, 3, 5)])
def test_linear_matches_torch_autograd_of_a_gather_dequantization(g, M, B):
    rng = np.random.default_rng(20 + g + M + B)
    C_out, G, N = 6, 5, 7
    cb, codes, s = _layer(rng, C_out, G, g, M, B)
    x = rng.normal(size=(N, G * g))
    dy = rng.normal(size=(N, C_out))
    dC = O.codebook_grad(_spec(g, M, B), {"codes": codes, "scales": s, "x": x}, dy)
    C_t = torch.tensor(cb, dtype=torch.float64, requires_grad=True)
    idx = torch.from_numpy(codes.astype(np.int64))
    parts = [C_t[m][idx[:, :, m]] for m in range(M)]           # [C_out, G, g] each
    W = torch.stack(parts).sum(0).reshape(C_out, G * g) * torch.from_numpy(s.astype(np.float64))[:, None]
    y = torch.from_numpy(x) @ W.T
    (y * torch.from_numpy(dy)).sum().backward()
    np.testing.assert_allclose(dC, C_t.grad.numpy(), rtol=1e-11, atol=1e-11)


@pytest.mark.parametrize("C,C_out,H,Wd,kh,kw,stride,pad,g", [
    (2, 3, 5, 4, 3, 3, 1, 1, 9),
    (3, 2, 6, 6, 3, 3, 2, 1, 3),
    (4, 3, 3, 5, 1, 1, 1, 0, 4),
    (8, 4, 5, 5, 3, 3, 1, 1, 8),
])
def test_conv_weight_gradient_matches_torch_autograd(C, C_out, H, Wd, kh, kw, stride, pad, g):
    """dW of the im2col convolution equals torch's conv2d weight gradient."""
    rng = np.random.default_rng(C * 10 + H + kh)
    x = rng.normal(size=(2, C, H, Wd))
    OH = (H + 2 * pad - kh) // stride + 1
    OW = (Wd + 2 * pad - kw) // stride + 1
    dy = rng.normal(size=(2, C_out, OH, OW))
    dW = O.weight_grad_conv(x, dy, kh, kw, stride, pad)
    W4 = torch.zeros((C_out, C, kh, kw), dtype=torch.float64, requires_grad=True)
    y = torch.nn.functional.conv2d(torch.from_numpy(x), W4, stride=stride, padding=pad)
    (y * torch.from_numpy(dy)).sum().backward()
    np.testing.assert_allclose(dW, W4.grad.numpy().reshape(C_out, -1), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("g,M,B,C,kh,stride", [(9, 2, 3, 3, 3, 1), (8, 2, 4, 8, 3, 1), (4, 3, 2, 4, 1, 1), (3, 1, 5, 3, 3, 2)])
def test_conv_adjoint_identity(g, M, B, C, kh, stride):
    """<dC, V> = L(V) for random V: the gradient of the linear loss is its adjoint."""
    rng = np.random.default_rng(40 + g + C + stride)
    C_out, H, Wd = 3, 6, 5
    pad = kh // 2
    G = C * kh * kh // g
    cb, codes, s = _layer(rng, C_out, G, g, M, B)
    x = rng.normal(size=(2, C, H, Wd))
    OH = (H + 2 * pad - kh) // stride + 1
    OW = (Wd + 2 * pad - kh) // stride + 1
    dy = rng.normal(size=(2, C_out, OH, OW))
    spec = _spec(g, M, B, _conv(kh, kh, stride, pad))
    dC = O.codebook_grad(spec, {"codes": codes, "scales": s, "x": x}, dy)
    for _ in range(3):
        V = rng.normal(size=cb.shape)
        lhs = float(np.sum(dC * V))
        rhs = _loss(spec, V, codes, s, x, dy)
        assert abs(lhs - rhs) <= 1e-11 * (1 + abs(rhs))


def test_stored_dtypes_widen_exactly():
    """fp16 / bf16 inputs and gradients give the same result as their exact fp64 values."""
    rng = np.random.default_rng(50)
    g, M, B, C_out, G, N = 8, 2, 3, 4, 2, 6
    _, codes, s = _layer(rng, C_out, G, g, M, B)
    x16 = rng.normal(size=(N, G * g)).astype(np.float16)
    dy16 = rng.normal(size=(N, C_out)).astype(np.float16)
    spec = _spec(g, M, B)
    a = O.codebook_grad(spec, {"codes": codes, "scales": s, "x": x16}, dy16, x_dtype="f16", dy_dtype="f16")
    b = O.codebook_grad(spec, {"codes": codes, "scales": s, "x": x16.astype(np.float64)},
                        dy16.astype(np.float64), x_dtype="f32")
    assert np.array_equal(a, b)
    xb = O.f32_to_bf16_bits(x16.astype(np.float32))
    dyb = O.f32_to_bf16_bits(dy16.astype(np.float32))
    c = O.codebook_grad(spec, {"codes": codes, "scales": s, "x": xb}, dyb, x_dtype="bf16", dy_dtype="bf16")
    xr = O.bf16_bits_to_f32(xb).astype(np.float64)
    dyr = O.bf16_bits_to_f32(dyb).astype(np.float64)
    d = O.codebook_grad(spec, {"codes": codes, "scales": s, "x": xr}, dyr, x_dtype="f32")
    assert np.array_equal(c, d)


@pytest.mark.parametrize("conv", [None, (3, 1, 1), (1, 1, 0), (3, 2, 1)])
def test_entry_sampled_gradient_matches_full(conv):
    """The per-entry evaluation used at full layer sizes agrees with the whole-tensor oracle."""
    rng = np.random.default_rng(60 + (0 if conv is None else conv[0] + conv[1]))
    g, M, B, C_out = 8, 2, 3, 5
    if conv is None:
        G, N = 4, 9
        x = rng.normal(size=(N, G * g))
        dy = rng.normal(size=(N, C_out))
        spec = _spec(g, M, B)
    else:
        kh, stride, pad = conv
        C, H, Wd = 8, 5, 6
        G = C * kh * kh // g
        x = rng.normal(size=(2, C, H, Wd))
        OH = (H + 2 * pad - kh) // stride + 1
        OW = (Wd + 2 * pad - kh) // stride + 1
        dy = rng.normal(size=(2, C_out, OH, OW))
        spec = _spec(g, M, B, _conv(kh, kh, stride, pad))
    _, codes, s = _layer(rng, C_out, G, g, M, B)
    inputs = {"codes": codes, "scales": s, "x": x}
    full = O.codebook_grad(spec, inputs, dy)
    entries = [(m, k) for m in range(M) for k in range(1 << B)]
    part = O.codebook_grad_entries(spec, inputs, dy, entries)
    np.testing.assert_allclose(part, full.reshape(-1, g), rtol=1e-12, atol=1e-12)
