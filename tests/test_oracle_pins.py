"""Pins of the fp64 oracle against things other than itself.

Each test checks the oracle against brute force on tiny inputs, a closed form,
an exact invariant, or an independent library routine, so that a dropped
term, a wrong index or a transposed operand in the oracle fails here.
"""
import itertools
import math

import numpy as np
import pytest
import torch

import oracle as O


def _rand_layer(rng, C_out, G, g, M, B, N):
    cb = rng.normal(0.0, 0.1, size=(M, 1 << B, g))
    codes = rng.integers(0, 1 << B, size=(C_out, G, M))
    codes = codes.astype(np.uint8 if B <= 8 else np.uint16)
    s = rng.uniform(0.5, 1.5, size=C_out).astype(np.float32)
    x = rng.normal(0.0, 1.0, size=(N, G * g))
    return cb, codes, s, x


def _brute_linear(x, cb, codes, s, g):
    """y[n, i] = fsum over (j, m, t) of x[n, j*g+t] * s_i * C[m, b_ijm, t]; no W is formed."""
    N = x.shape[0]
    C_out, G, M = codes.shape
    y = np.zeros((N, C_out))
    for n in range(N):
        for i in range(C_out):
            terms = []
            for j in range(G):
                for m in range(M):
                    b = int(codes[i, j, m])
                    for t in range(g):
                        terms.append(float(x[n, j * g + t]) * float(s[i]) * float(cb[m, b, t]))
            y[n, i] = math.fsum(terms)
    return y


@pytest.mark.parametrize("g,M,B", [(1, 1, 1), (2, 3, 2), (8, 2, 8), (9, 4, 5), (8, 1, 16), (4, 2, 3), (16, 3, 8)])
def test_linear_matches_brute_force(g, M, B):
    rng = np.random.default_rng(100 + g * 31 + M * 7 + B)
    C_out, G, N = 5, 4, 3
    cb, codes, s, x = _rand_layer(rng, C_out, G, g, M, B, N)
    cb32 = cb.astype(np.float32)
    W = O.dequantize(cb32, codes, s, g, "f32")
    y = O.linear_forward(x, W)
    y_ref = _brute_linear(x, cb32.astype(np.float64), codes, s.astype(np.float64), g)
    assert np.max(np.abs(y - y_ref)) <= 1e-13 * np.max(np.abs(y_ref))


def test_dequantize_elementwise_definition():
    """W[i, j*g+t] == s_i * sum_m C[m, b_ijm, t], element by element."""
    rng = np.random.default_rng(7)
    g, M, B, C_out, G = 3, 3, 4, 4, 5
    cb, codes, s, _ = _rand_layer(rng, C_out, G, g, M, B, 1)
    W = O.dequantize(cb.astype(np.float32), codes, s, g, "f32")
    for i in range(C_out):
        for j in range(G):
            for t in range(g):
                v = float(s[i]) * math.fsum(float(np.float32(cb[m, codes[i, j, m], t])) for m in range(M))
                assert W[i, j * g + t] == pytest.approx(v, rel=1e-15, abs=1e-300)


def test_one_hot_codebook_reduces_to_gather():
    """M=1, C[k][t] = [t == k mod g]: each group contributes x at offset (b mod g)."""
    rng = np.random.default_rng(11)
    g, B, C_out, G, N = 8, 4, 7, 6, 5
    k = np.arange(1 << B)
    cb = (np.arange(g)[None, :] == (k % g)[:, None]).astype(np.float32)[None]   # [1, 2^B, g]
    codes = rng.integers(0, 1 << B, size=(C_out, G, 1)).astype(np.uint8)
    s = rng.choice([0.5, 1.0, 2.0], size=C_out).astype(np.float32)
    x = rng.integers(-50, 50, size=(N, G * g)).astype(np.float64)    # exact arithmetic
    y = O.linear_forward(x, O.dequantize(cb, codes, s, g, "f32"))
    # plain gather: column index j*g + (b mod g)
    col = np.arange(G)[None, :] * g + (codes[:, :, 0].astype(np.int64) % g)  # [C_out, G]
    gathered = np.take_along_axis(x[:, None, :].repeat(C_out, 1), col[None, :, :].repeat(N, 0), axis=2)
    y_ref = gathered.sum(axis=2) * s[None, :].astype(np.float64)
    assert np.array_equal(y, y_ref)


def test_codebook_power_of_two_scaling_is_exact():
    rng = np.random.default_rng(12)
    cb, codes, s, x = _rand_layer(rng, 6, 5, 8, 2, 6, 4)
    cb = cb.astype(np.float32)
    y1 = O.linear_forward(x, O.dequantize(cb, codes, s, 8, "f32"))
    y2 = O.linear_forward(x, O.dequantize(cb * np.float32(4.0), codes, s, 8, "f32"))
    assert np.array_equal(y2, 4.0 * y1)


def test_scale_is_per_output_column():
    rng = np.random.default_rng(13)
    cb, codes, s, x = _rand_layer(rng, 6, 5, 8, 2, 6, 4)
    cb = cb.astype(np.float32)
    ones = np.ones_like(s)
    y1 = O.linear_forward(x, O.dequantize(cb, codes, ones, 8, "f32"))
    ys = O.linear_forward(x, O.dequantize(cb, codes, s, 8, "f32"))
    np.testing.assert_allclose(ys, y1 * s[None, :].astype(np.float64), rtol=1e-13, atol=1e-13)
    # the scale multiplies output rows of W, not the codeword sum per input:
    # a unit scale on one channel leaves that output column unchanged
    s2 = s.copy()
    s2[2] = 1.0
    y2 = O.linear_forward(x, O.dequantize(cb, codes, s2, 8, "f32"))
    assert np.array_equal(y2[:, 2], y1[:, 2])


def test_codebook_additivity_and_permutation():
    rng = np.random.default_rng(14)
    M = 3
    cb, codes, s, x = _rand_layer(rng, 5, 4, 8, M, 5, 3)
    cb = cb.astype(np.float32)
    y = O.linear_forward(x, O.dequantize(cb, codes, s, 8, "f32"))
    parts = sum(O.linear_forward(x, O.dequantize(cb[m:m + 1], codes[:, :, m:m + 1], s, 8, "f32")) for m in range(M))
    np.testing.assert_allclose(y, parts, rtol=1e-12, atol=1e-12)
    perm = [2, 0, 1]
    yp = O.linear_forward(x, O.dequantize(cb[perm], codes[:, :, perm], s, 8, "f32"))
    np.testing.assert_allclose(y, yp, rtol=1e-12, atol=1e-12)


def test_group_order_along_k():
    """Swapping two groups' codes must move the contribution to other inputs."""
    rng = np.random.default_rng(15)
    cb, codes, s, x = _rand_layer(rng, 3, 4, 8, 2, 5, 2)
    cb = cb.astype(np.float32)
    W = O.dequantize(cb, codes, s, 8, "f32")
    codes2 = codes.copy()
    codes2[:, [0, 1], :] = codes[:, [1, 0], :]
    W2 = O.dequantize(cb, codes2, s, 8, "f32")
    assert np.array_equal(W[:, 0:8], W2[:, 8:16]) and np.array_equal(W[:, 8:16], W2[:, 0:8])


def _brute_conv(x, W4, stride, pad):
    n, C, H, Wd = x.shape
    C_out, _, kh, kw = W4.shape
    OH = (H + 2 * pad - kh) // stride + 1
    OW = (Wd + 2 * pad - kw) // stride + 1
    y = np.zeros((n, C_out, OH, OW))
    for b in range(n):
        for o in range(C_out):
            for oh in range(OH):
                for ow in range(OW):
                    terms = []
                    for c in range(C):
                        for r in range(kh):
                            for q in range(kw):
                                ih, iw = oh * stride - pad + r, ow * stride - pad + q
                                if 0 <= ih < H and 0 <= iw < Wd:
                                    terms.append(float(x[b, c, ih, iw]) * float(W4[o, c, r, q]))
                    y[b, o, oh, ow] = math.fsum(terms)
    return y


@pytest.mark.parametrize("C,C_out,H,Wd,kh,kw,stride,pad,g", [
    (2, 3, 5, 4, 3, 3, 1, 1, 9),
    (3, 2, 6, 6, 3, 3, 2, 1, 3),
    (4, 3, 3, 5, 1, 1, 1, 0, 4),
    (2, 2, 4, 5, 2, 3, 1, 0, 6),
    (8, 4, 5, 5, 3, 3, 1, 1, 8),   # g=8 groups straddle channel boundaries
])
def test_conv_im2col_matches_direct_conv(C, C_out, H, Wd, kh, kw, stride, pad, g):
    rng = np.random.default_rng(C * 100 + H)
    K = C * kh * kw
    G = K // g
    cb, codes, s, _ = _rand_layer(rng, C_out, G, g, 2, 4, 1)
    cb = cb.astype(np.float32)
    W = O.dequantize(cb, codes, s, g, "f32")
    x = rng.normal(size=(2, C, H, Wd))
    y = O.conv_forward(x, W, kh, kw, stride, pad)
    W4 = W.reshape(C_out, C, kh, kw)
    y_ref = _brute_conv(x, W4, stride, pad)
    assert y.shape == y_ref.shape
    np.testing.assert_allclose(y, y_ref, rtol=1e-13, atol=1e-13)
    y_t = torch.nn.functional.conv2d(torch.from_numpy(x), torch.from_numpy(W4), stride=stride, padding=pad).numpy()
    np.testing.assert_allclose(y, y_t, rtol=1e-12, atol=1e-12)


def test_forward_sampled_matches_full():
    from workloads import LayerSpec, ConvGeom, generate
    for spec in [
        LayerSpec(name="c", C_out=16, K=72, g=8, M=2, B=6, n=2, conv=ConvGeom(8, 3, 3, 1, 1, 6, 5)),
        LayerSpec(name="c2", C_out=8, K=27, g=9, M=1, B=5, n=3, conv=ConvGeom(3, 3, 3, 2, 1, 7, 7)),
        LayerSpec(name="l", C_out=24, K=64, g=8, M=4, B=8, n=10, x_dtype="i8"),
    ]:
        inp = generate(spec, 5)
        y = O.forward(spec, inp)
        rng = np.random.default_rng(0)
        tok = rng.integers(0, spec.tokens, size=7)
        ch = rng.integers(0, spec.C_out, size=5)
        ys = O.forward_sampled(spec, inp, tok, ch)
        if spec.conv is None:
            full = y
        else:
            full = y.transpose(0, 2, 3, 1).reshape(spec.tokens, spec.C_out)
        np.testing.assert_allclose(ys, full[np.ix_(tok, ch)], rtol=1e-13, atol=1e-13)


def test_a8_activation_factorisation():
    rng = np.random.default_rng(16)
    cb, codes, s, _ = _rand_layer(rng, 6, 4, 8, 2, 8, 1)
    W = O.dequantize(cb.astype(np.float16), codes, s, 8, "f16")
    q = np.clip(np.rint(rng.normal(0, 30, size=(5, 32))), -127, 127).astype(np.int8)
    a = (rng.uniform(0.5, 1.5, size=5) / 127).astype(np.float32)
    y = O.linear_forward(O.activations_f64(q, "i8", a), W)
    y1 = O.linear_forward(O.activations_f64(q, "i8", np.ones(5, np.float32)), W)
    np.testing.assert_allclose(y, a[:, None].astype(np.float64) * y1, rtol=1e-13, atol=1e-15)
    # exactness of a*q in fp64
    X = O.activations_f64(q, "i8", a)
    for n in range(5):
        for k in range(0, 32, 7):
            assert X[n, k] == float(a[n]) * float(q[n, k])


def test_bf16_and_fp16_storage_widening():
    vals = np.array([1.0, -2.5, 3.140625, 1e-3, 65504.0], dtype=np.float32)
    bits = torch.from_numpy(vals).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    back = O.to_f64(bits, "bf16")
    ref = torch.from_numpy(vals).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(back, ref)


# ---------------------------------------------------------------------------
# Decode emulation (bit-exact reference for decoded tiles)
# ---------------------------------------------------------------------------

def _torch_decode(cb16, codes, s, g, tile, scaled):
    """Independent emulation with torch CPU tensors.

    fp16 tiles accumulate in torch.float16 (every add rounded to fp16);
    other tiles accumulate in float32.
    """
    idx = torch.from_numpy(codes.astype(np.int64))
    if tile == "f16":
        C = torch.from_numpy(cb16)
    else:
        C = torch.from_numpy(cb16.astype(np.float32))
    acc = C[0][idx[:, :, 0]]
    for m in range(1, C.shape[0]):
        acc = acc + C[m][idx[:, :, m]]
    acc = acc.float()
    if scaled:
        acc = acc * torch.from_numpy(s)[:, None, None]
    acc = acc.reshape(codes.shape[0], -1)
    if tile == "f16":
        return acc.to(torch.float16).numpy()
    if tile == "bf16":
        return acc.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    return acc.numpy()


@pytest.mark.parametrize("tile", ["f16", "bf16", "f32"])
@pytest.mark.parametrize("scaled", [True, False])
@pytest.mark.parametrize("M", [1, 2, 3, 4])
def test_decode_emulation_matches_torch_casts(tile, scaled, M):
    rng = np.random.default_rng(20 + M)
    B, g = 8, 8
    cb = rng.normal(0.0, 0.05, size=(M, 1 << B, g))
    cb[:, :8, :] *= 1e-4         # push some sums into the fp16 subnormal range
    cb16 = cb.astype(np.float16)
    codes = rng.integers(0, 1 << B, size=(40, 12, M)).astype(np.uint8)
    codes[:4] = rng.integers(0, 8, size=(4, 12, M))      # sums of tiny codewords only
    s = rng.uniform(0.5, 1.5, size=40).astype(np.float32)
    got = O.decode_emulate(cb16, codes, s, g, "f16", tile, scaled)
    ref = _torch_decode(cb16, codes, s, g, tile, scaled)
    if tile == "f16":
        assert np.array_equal(got.view(np.uint16), ref.view(np.uint16))
        assert np.any(np.abs(got) < np.float16(6.1e-5))     # subnormals exercised
    else:
        assert np.array_equal(got.view(np.uint32) if tile == "f32" else got,
                              ref.view(np.uint32) if tile == "f32" else ref)


def _adversarial_f16_pairs(rng, n):
    """fp16 pairs spanning every exponent gap, both signs, subnormals and ties."""
    e1 = rng.integers(-24, 16, size=n)
    e2 = e1 - rng.integers(0, 30, size=n)
    m1 = rng.integers(1024, 2048, size=n)
    m2 = rng.integers(1024, 2048, size=n)
    a = (np.sign(rng.normal(size=n)) * m1 * np.exp2(e1 - 10.0)).astype(np.float16)
    b = (np.sign(rng.normal(size=n)) * m2 * np.exp2(np.maximum(e2, -24) - 10.0)).astype(np.float16)
    return a, b


def test_two_fp16_addends_round_once():
    """For two fp16 addends, rounding the fp32 sum to fp16 equals rounding the exact sum.

    The fp16-tile decode relies on this for M = 2: an fp16 add and an fp32
    add followed by one rounding give the same bits.  The exact sum is
    formed in fp64 (fp16 values have 11 significant bits within 40 binades).
    """
    rng = np.random.default_rng(123)
    a, b = _adversarial_f16_pairs(rng, 400000)
    exact = a.astype(np.float64) + b.astype(np.float64)
    once = exact.astype(np.float16)                   # one rounding of the exact value
    via32 = (a.astype(np.float32) + b.astype(np.float32)).astype(np.float16)
    assert np.array_equal(once.view(np.uint16), via32.view(np.uint16))
    # three addends can differ: the fp16 chain is a distinct rule for M >= 3
    c = (rng.normal(0, 0.05, size=200000)).astype(np.float16)
    x = rng.normal(0, 0.05, size=200000).astype(np.float16)
    y = rng.normal(0, 0.05, size=200000).astype(np.float16)
    chain = ((x.astype(np.float32) + y.astype(np.float32)).astype(np.float16).astype(np.float32)
             + c.astype(np.float32)).astype(np.float16)
    f32 = (x.astype(np.float32) + y.astype(np.float32) + c.astype(np.float32)).astype(np.float16)
    assert np.any(chain.view(np.uint16) != f32.view(np.uint16))


def test_bf16_rounding_ties_and_carries():
    # exact ties between bf16 neighbours, both parities, and a mantissa carry
    pats = np.array([0x3F808000, 0x3F818000, 0x3F7FFFFF, 0x3F80FFFF, 0x00018000, 0xBF808001], dtype=np.uint32)
    f = pats.view(np.float32)
    got = O.f32_to_bf16_bits(f)
    ref = torch.from_numpy(f.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got, ref)


def test_decode_emulation_against_float_definition():
    """fp32 rule: the decoded value is within half an fp16 ulp of the exact scaled weight."""
    rng = np.random.default_rng(21)
    M, B, g = 4, 8, 8
    cb32 = rng.normal(0, 0.05, size=(M, 1 << B, g)).astype(np.float16).astype(np.float32)
    codes = rng.integers(0, 256, size=(30, 10, M)).astype(np.uint8)
    s = rng.uniform(0.5, 1.5, size=30).astype(np.float32)
    W = O.dequantize(cb32, codes, s, g, "f32")
    d = O.decode_emulate(cb32, codes, s, g, "f32", "f16", True).astype(np.float64)
    ulp = np.spacing(np.abs(d.astype(np.float16))).astype(np.float64)
    assert np.all(np.abs(d - W) <= 0.5 * ulp + 4 * np.abs(W) * 2.0 ** -24)


def test_fp16_chain_rounds_each_partial_sum_once():
    """fp16 rule: every partial sum is the correctly rounded fp16 sum of the previous one and a codeword."""
    rng = np.random.default_rng(22)
    M, B, g = 4, 8, 8
    cb16 = rng.normal(0, 0.05, size=(M, 1 << B, g)).astype(np.float16)
    codes = rng.integers(0, 256, size=(30, 10, M)).astype(np.uint8)
    s = np.ones(30, dtype=np.float32)
    d = O.decode_emulate(cb16, codes, s, g, "f16", "f16", False).astype(np.float64).reshape(30, 10, g)
    # re-derive the chain in fp64 with one explicit rounding per step
    part = cb16[0][codes[:, :, 0]].astype(np.float64)
    bound = np.zeros_like(part)
    for m in range(1, M):
        exact = part + cb16[m][codes[:, :, m]].astype(np.float64)   # exact in fp64
        part = exact.astype(np.float16).astype(np.float64)
        bound += 0.5 * np.spacing(np.abs(part).astype(np.float16)).astype(np.float64)
    assert np.array_equal(d, part)
    total = sum(cb16[m][codes[:, :, m]].astype(np.float64) for m in range(M))
    assert np.all(np.abs(d - total) <= bound + 1e-12)


# ---------------------------------------------------------------------------
# Appendix FLOP count and breakpoint
# ---------------------------------------------------------------------------

def _lut_route_conv_counting(x, cb, codes, kh, kw):
    """The appendix rearrangement, written out with explicit op counting.

    One group per (output, input) channel filter (g = kh*kw), stride 1, 'same'
    zero padding.  Every input channel is convolved with every codeword of every
    codebook (the LUT), then each output channel sums the code-indexed maps.
    """
    n, C_in, H, Wd = x.shape
    M, K2, g = cb.shape
    C_out = codes.shape[0]
    pad = (kh - 1) // 2
    mults = adds = 0
    lut = np.zeros((M, K2, C_in, H, Wd))
    for m in range(M):
        for k in range(K2):
            filt = cb[m, k].reshape(kh, kw)
            for c in range(C_in):
                for oh in range(H):
                    for ow in range(Wd):
                        acc = None
                        for r in range(kh):
                            for q in range(kw):
                                ih, iw = oh - pad + r, ow - pad + q
                                v = x[0, c, ih, iw] if (0 <= ih < H and 0 <= iw < Wd) else 0.0
                                p = v * filt[r, q]
                                mults += 1
                                if acc is None:
                                    acc = p
                                else:
                                    acc = acc + p
                                    adds += 1
                        lut[m, k, c, oh, ow] = acc
    y = np.zeros((1, C_out, H, Wd))
    for i in range(C_out):
        for c in range(C_in):
            for m in range(M):
                y[0, i] += lut[m, codes[i, c, m], c]
                adds += H * Wd
    return y, mults, adds


def test_appendix_flop_count_and_lut_route():
    rng = np.random.default_rng(30)
    M, k, C_in, C_out, H, Wd = 2, 2, 3, 4, 4, 3
    kh = kw = 3
    cb = rng.normal(size=(M, 1 << k, kh * kw))
    codes = rng.integers(0, 1 << k, size=(C_out, C_in, M)).astype(np.uint8)
    x = rng.normal(size=(1, C_in, H, Wd))
    ones = np.ones(C_out, dtype=np.float32)
    W = O.dequantize(cb.astype(np.float32), codes, ones, kh * kw, "f32")
    y_def = O.conv_forward(x, W, kh, kw, 1, 1)
    y_lut, mults, adds = _lut_route_conv_counting(x, cb.astype(np.float32).astype(np.float64), codes, kh, kw)
    np.testing.assert_allclose(y_lut, y_def, rtol=1e-12, atol=1e-12)
    # the count of eq. (13) (the gather additions start from a zero map: one add per term)
    assert mults + adds == O.lut_conv_flops(M, k, C_in, C_out, H, Wd, kh, kw)
    assert O.dense_conv_flops(C_out, C_in, H, Wd, kh, kw) == 2 * y_def.size * C_in * kh * kw


@pytest.mark.parametrize("M,k", [(1, 8), (2, 8), (4, 8), (2, 4)])
def test_breakpoint_follows_count(M, k):
    bp = O.lut_breakpoint_cout(M, k, 9)
    C_in, h, w = 5, 7, 6
    lo, hi = math.floor(bp), math.floor(bp) + 1
    if lo != bp:
        assert O.lut_conv_flops(M, k, C_in, lo, h, w, 3, 3) > O.dense_conv_flops(lo, C_in, h, w, 3, 3)
    assert O.lut_conv_flops(M, k, C_in, hi, h, w, 3, 3) < O.dense_conv_flops(hi, C_in, h, w, 3, 3)
    assert bp == pytest.approx(17 * M * 2 ** k / (18 - M))


def test_error_metric():
    y_ref = np.array([[1.0, -4.0], [2.0, 0.5]])
    y = y_ref + np.array([[0.0, 0.004], [-0.002, 0.0]])
    assert O.rel_err_inf(y, y_ref) == pytest.approx(0.001)


# ---------------------------------------------------------------------------
# O6: RMS-relative and floored per-element errors, and the rounding bound
# ---------------------------------------------------------------------------

def test_rms_and_elementwise_errors_closed_forms():
    rng = np.random.default_rng(12)
    y = rng.normal(size=(40, 7))
    # a uniform relative perturbation eps gives exactly eps in both forms
    assert math.isclose(O.rel_err_rms(y * 1.003, y), 0.003, rel_tol=1e-9)
    assert math.isclose(O.rel_err_elem(y * 1.003, y), 0.003, rel_tol=1e-9)
    # a constant offset c gives c / rms(y) in RMS form
    rms = math.sqrt(float(np.mean(y * y)))
    assert math.isclose(O.rel_err_rms(y + 0.01, y), 0.01 / rms, rel_tol=1e-9)
    # one element near zero: judged against the floor, not against its own magnitude
    z = y.copy()
    z[3, 2] = 1e-9
    w = z.copy()
    w[3, 2] += 1e-4
    assert math.isclose(O.rel_err_elem(w, z), 1e-4 / (1e-3 * math.sqrt(float(np.mean(z * z)))), rel_tol=1e-9)
    # a localised error the infinity norm over the whole output dilutes
    v = y.copy()
    v[:, 0] *= 1e-3
    u = v.copy()
    u[5, 0] *= 2.0
    assert O.rel_err_inf(u, v) < 2e-3 < O.rel_err_elem(u, v)


def test_abs_inputs_forward_is_sum_of_magnitudes():
    """forward(abs_inputs) == fsum over (k, m) of |x_k| s_i |C_m[b][t]|, brute force; it dominates |Y*|."""
    rng = np.random.default_rng(13)
    g, M, B, C_out, G, N = 4, 3, 4, 5, 3, 4
    cb, codes, s, x = _rand_layer(rng, C_out, G, g, M, B, N)
    from workloads import LayerSpec
    spec = LayerSpec(name="abs", C_out=C_out, K=G * g, g=g, M=M, B=B, n=N, codebook_dtype="f32", x_dtype="f32",
                     y_dtype="f32", tile_dtype="f32")
    inp = {"codebooks": cb.astype(np.float32), "codes": codes, "scales": s, "x": x.astype(np.float32),
           "x_scales": None}
    a = O.forward(spec, O.abs_inputs(spec, inp))
    for n in range(N):
        for i in range(C_out):
            terms = [abs(float(inp["x"][n, j * g + t])) * float(s[i]) * abs(float(inp["codebooks"][m, codes[i, j, m], t]))
                     for j in range(G) for m in range(M) for t in range(g)]
            assert math.isclose(a[n, i], math.fsum(terms), rel_tol=1e-13)
    assert np.all(a >= np.abs(O.forward(spec, inp)) * (1 - 1e-13))


def _emulated_gpu_forward(spec, inp):
    """The decode path's arithmetic written out in numpy: fp16 tile weights
    (unscaled, decode emulation), products and sums in fp32, scale on the fp32
    sum, one rounding to the output dtype."""
    wt = O.decode_emulate(inp["codebooks"], inp["codes"], inp["scales"], spec.g, spec.codebook_dtype,
                          spec.tile_dtype, scaled=False).astype(np.float32)
    x = inp["x"].astype(np.float32)
    acc = (x @ wt.T).astype(np.float32)
    y = (acc * inp["scales"].astype(np.float32)[None, :]).astype(np.float32)
    return y.astype(np.float16 if spec.y_dtype == "f16" else np.float32).astype(np.float64)


@pytest.mark.parametrize("M", [1, 2, 4])
def test_rounding_bound_holds_for_emulated_arithmetic_and_catches_one_wrong_element(M):
    from workloads import LayerSpec, generate
    spec = LayerSpec(name="bound", C_out=48, K=256, g=8, M=M, B=8, n=200)
    inp = generate(spec, 21 + M)
    y_ref = O.forward(spec, inp)
    a_ref = O.forward(spec, O.abs_inputs(spec, inp))
    bound = O.rounding_bound(spec, y_ref, a_ref, "decode")
    y = _emulated_gpu_forward(spec, inp)
    assert np.all(np.abs(y - y_ref) <= bound)
    # the bound stays a small fraction of the output's scale, and an error of
    # twice the bound in one element is flagged there and nowhere else
    rms = math.sqrt(float(np.mean(y_ref * y_ref)))
    assert float(np.max(bound)) < 0.1 * rms
    bad = y.copy()
    bad[17, 5] += 2.0 * bound[17, 5]
    viol = np.argwhere(np.abs(bad - y_ref) > bound)
    assert [tuple(v) for v in viol] == [(17, 5)]
    # a swapped pair of output channels (a plausible indexing mistake) is caught
    sw = y.copy()
    sw[:, [3, 4]] = sw[:, [4, 3]]
    assert np.any(np.abs(sw - y_ref) > bound)
