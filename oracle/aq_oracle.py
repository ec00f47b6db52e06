"""Plain fp64 CPU oracle of the AQ linear / im2col-convolution forward and of
its codebook gradient.

TEST INFRASTRUCTURE ONLY: imported by tests, by the smoke check and by the
benchmark's CPU-baseline leg, never by the GPU library.

What is computed (paper: "AQUATIC-Diff", Sec. 2.4 eq. (4), Sec. 3.1.1, and
the appendix proof of FLOPs savings):

* A weight matrix is split along its input dimension into groups of ``g``
  consecutive weights.  Group ``j`` of output row ``i`` stores ``M`` integer
  codes ``b[i, j, m]``; the group is reconstructed as the sum over ``m`` of
  codeword ``b[i, j, m]`` of codebook ``m`` (eq. (4): groups concatenated in
  order, each the sum of its M selected codebook rows).
* Each output row then carries one fp32 scale ``s[i]`` multiplied after the
  codeword sum (the paper's eq. (4) has no scale; the per-output-channel
  scale is part of the layer format used here).
* A linear layer computes ``Y = X W^T`` with tokens as rows (the paper writes
  ``Y = W X`` with tokens as columns; this is its transpose).
* A convolution is lowered by im2col (Sec. 3.1.1): each output position
  becomes a token whose input vector runs over (input channel, kernel row,
  kernel column) with the channel outermost, the order of a PyTorch weight
  tensor ``[C_out, C_in, kh, kw]`` flattened per output channel.

Every stored value (fp32, fp16, bf16, int8) converts to fp64 exactly, and the
arithmetic is fp64 with numpy's BLAS matmul as the one library primitive.
The LUT route of the appendix (eq. (12)) is an exact algebraic rearrangement
of the same sum, so this plain definition is also the oracle for it.

The codebook gradient (O7 below; the continuous step of PV-Tuning, Sec. 3.2)
is the chain rule through the same definitions: dW = dY^T X, then a
scatter-add of s[i] * dW over the codes.
"""
from __future__ import annotations

from typing import Optional, Sequence

import numpy as np


# ---------------------------------------------------------------------------
# Storage dtypes -> fp64
# ---------------------------------------------------------------------------

def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """bf16 stored as uint16 bit patterns -> float32 (exact: bf16 is fp32's top half)."""
    b = np.asarray(bits).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32)


def to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact widening of a stored array to fp64."""
    if dtype == "bf16":
        return bf16_bits_to_f32(a).astype(np.float64)
    if dtype in ("f32", "f16", "i8"):
        return np.asarray(a).astype(np.float64)
    raise ValueError(dtype)


# ---------------------------------------------------------------------------
# O1: dequantization (eq. (4) plus the per-output-channel scale)
# ---------------------------------------------------------------------------

def dequantize(codebooks: np.ndarray, codes: np.ndarray, scales: np.ndarray, g: int,
               codebook_dtype: str = "f32") -> np.ndarray:
    """Dense weight matrix W [C_out, K] in fp64.

    ``codebooks`` is [M, 2**B, g], ``codes`` is [C_out, G, M] and ``scales`` is
    [C_out].  W[i, j*g + t] = s[i] * sum_m C[m, b[i, j, m], t].
    """
    C = to_f64(codebooks, codebook_dtype)
    M, _, gg = C.shape
    if gg != g:
        raise ValueError("codebook row length must equal the group size g")
    C_out, G, M2 = codes.shape
    if M2 != M:
        raise ValueError("codes and codebooks disagree on M")
    idx = codes.astype(np.int64)
    group_sum = np.zeros((C_out, G, g), dtype=np.float64)
    for m in range(M):
        group_sum += C[m][idx[:, :, m]]          # [C_out, G, g]
    W = group_sum.reshape(C_out, G * g)          # groups concatenated along K
    return np.asarray(scales, dtype=np.float64)[:, None] * W


# ---------------------------------------------------------------------------
# Activations (A8: x = a_n * q, per-token scale)
# ---------------------------------------------------------------------------

def activations_f64(x: np.ndarray, x_dtype: str, x_scales: Optional[np.ndarray] = None) -> np.ndarray:
    """Activations in fp64; int8 inputs are dequantized with their per-token scale.

    The product a_n * q is exact in fp64 (7-bit integer times a 24-bit
    significand).
    """
    X = to_f64(x, x_dtype)
    if x_dtype == "i8":
        if x_scales is None:
            raise ValueError("int8 activations need per-token scales")
        a = np.asarray(x_scales, dtype=np.float64)
        X = X * a.reshape((-1,) + (1,) * (X.ndim - 1))
    return X


# ---------------------------------------------------------------------------
# O2 / O3: linear and im2col convolution
# ---------------------------------------------------------------------------

def linear_forward(X: np.ndarray, W: np.ndarray) -> np.ndarray:
    """Y [N, C_out] = X [N, K] @ W[C_out, K]^T in fp64."""
    return np.asarray(X, dtype=np.float64) @ np.asarray(W, dtype=np.float64).T


def im2col(x: np.ndarray, kh: int, kw: int, stride: int, pad: int) -> np.ndarray:
    """NCHW input -> [n*OH*OW, C*kh*kw] with zero padding (Sec. 3.1.1).

    Rows run over (image, output row, output column); columns over
    (channel, kernel row, kernel column), channel outermost.
    """
    x = np.asarray(x, dtype=np.float64)
    n, C, H, W = x.shape
    OH = (H + 2 * pad - kh) // stride + 1
    OW = (W + 2 * pad - kw) // stride + 1
    xp = np.zeros((n, C, H + 2 * pad, W + 2 * pad), dtype=np.float64)
    xp[:, :, pad:pad + H, pad:pad + W] = x
    cols = np.empty((n, OH, OW, C, kh, kw), dtype=np.float64)
    for r in range(kh):
        for s in range(kw):
            patch = xp[:, :, r:r + stride * (OH - 1) + 1:stride, s:s + stride * (OW - 1) + 1:stride]
            cols[:, :, :, :, r, s] = patch.transpose(0, 2, 3, 1)
    return cols.reshape(n * OH * OW, C * kh * kw)


def conv_forward(x: np.ndarray, W: np.ndarray, kh: int, kw: int, stride: int, pad: int) -> np.ndarray:
    """Convolution as im2col + matmul; returns NCHW [n, C_out, OH, OW] fp64."""
    n, C, H, Wd = x.shape
    OH = (H + 2 * pad - kh) // stride + 1
    OW = (Wd + 2 * pad - kw) // stride + 1
    cols = im2col(x, kh, kw, stride, pad)
    Y = cols @ np.asarray(W, dtype=np.float64).T             # [n*OH*OW, C_out]
    return Y.reshape(n, OH, OW, -1).transpose(0, 3, 1, 2).copy()


def forward(spec, inputs) -> np.ndarray:
    """Whole-layer forward for a layer description ``spec``.

    ``spec`` needs the attributes g, codebook_dtype, x_dtype and ``conv`` (None
    for a linear layer, else an object with kh, kw, stride, pad); ``inputs``
    holds codebooks, codes, scales, x and x_scales.
    """
    W = dequantize(inputs["codebooks"], inputs["codes"], inputs["scales"], spec.g, spec.codebook_dtype)
    X = activations_f64(inputs["x"], spec.x_dtype, inputs.get("x_scales"))
    if spec.conv is None:
        return linear_forward(X, W)
    c = spec.conv
    return conv_forward(X, W, c.kh, c.kw, c.stride, c.pad)


def forward_sampled(spec, inputs, tokens: Sequence[int], channels: Sequence[int]) -> np.ndarray:
    """Y*[tokens, channels] for a subset of outputs, without the full matmul.

    Tokens are flat indices into the token-major output (for a convolution,
    token = (b*OH + oh)*OW + ow).  Returns [len(tokens), len(channels)].
    """
    tokens = np.asarray(tokens, dtype=np.int64)
    channels = np.asarray(channels, dtype=np.int64)
    codes = inputs["codes"][channels]
    W = dequantize(inputs["codebooks"], codes, inputs["scales"][channels], spec.g, spec.codebook_dtype)
    if spec.conv is None:
        xs = inputs["x"][tokens]
        a = None if inputs.get("x_scales") is None else inputs["x_scales"][tokens]
        X = activations_f64(xs, spec.x_dtype, a)
        return X @ W.T
    c = spec.conv
    x = activations_f64(inputs["x"], spec.x_dtype, inputs.get("x_scales"))
    n, C, H, Wd = x.shape
    OH = (H + 2 * c.pad - c.kh) // c.stride + 1
    OW = (Wd + 2 * c.pad - c.kw) // c.stride + 1
    b = tokens // (OH * OW)
    oh = (tokens // OW) % OH
    ow = tokens % OW
    rows = np.zeros((len(tokens), C, c.kh, c.kw), dtype=np.float64)
    for r in range(c.kh):
        for s in range(c.kw):
            ih = oh * c.stride - c.pad + r
            iw = ow * c.stride - c.pad + s
            ok = (ih >= 0) & (ih < H) & (iw >= 0) & (iw < Wd)
            vals = np.zeros((len(tokens), C), dtype=np.float64)
            vals[ok] = x[b[ok], :, ih[ok], iw[ok]]
            rows[:, :, r, s] = vals
    return rows.reshape(len(tokens), -1) @ W.T


# ---------------------------------------------------------------------------
# O5: decode emulation for bit-exact checks of decoded weight tiles
# ---------------------------------------------------------------------------

def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bits with round-to-nearest-even (finite inputs).

    Adds 0x7FFF plus the lowest kept bit, then truncates: the standard
    round-half-to-even by bias on the IEEE bit pattern.
    """
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return r.astype(np.uint16)


def decode_emulate(codebooks: np.ndarray, codes: np.ndarray, scales: np.ndarray, g: int,
                   codebook_dtype: str, tile_dtype: str, scaled: bool = True) -> np.ndarray:
    """Decoded weights [C_out, K] exactly as the decode kernels produce them.

    * fp16 codebooks with an fp16 tile: the M codewords accumulate in IEEE
      binary16 in ascending m, rounding to nearest even after every add.  For
      M <= 2 this equals the fp32 sum rounded once to fp16 (two fp16 addends
      never double-round), so only M >= 3 differs from the next rule.
    * otherwise: IEEE fp32 sum in ascending m (no fused multiply-add).
    Then, when ``scaled``, ``w = fl32(acc * s[i])``; then one
    round-to-nearest-even to the tile dtype.  Returns float16 / float32 arrays,
    or uint16 bf16 bit patterns.
    """
    M = np.asarray(codebooks).shape[0]
    C_out, G, _ = codes.shape
    idx = codes.astype(np.int64)
    if codebook_dtype == "f16" and tile_dtype == "f16":
        C16 = np.asarray(codebooks).astype(np.float16)
        acc16 = C16[0][idx[:, :, 0]]
        for m in range(1, M):
            # an fp16 add: exact fp32 sum of two fp16 values, rounded once to fp16
            acc16 = (acc16.astype(np.float32) + C16[m][idx[:, :, m]].astype(np.float32)).astype(np.float16)
        acc = acc16.astype(np.float32)
    else:
        if codebook_dtype == "bf16":
            C = bf16_bits_to_f32(codebooks)
        else:
            C = np.asarray(codebooks).astype(np.float32)
        acc = C[0][idx[:, :, 0]].astype(np.float32)
        for m in range(1, M):
            acc = (acc + C[m][idx[:, :, m]]).astype(np.float32)
    if scaled:
        acc = (acc * np.asarray(scales, dtype=np.float32)[:, None, None]).astype(np.float32)
    acc = acc.reshape(C_out, G * g)
    if tile_dtype == "f32":
        return acc
    if tile_dtype == "f16":
        return acc.astype(np.float16)
    if tile_dtype == "bf16":
        return f32_to_bf16_bits(acc)
    raise ValueError(tile_dtype)


# ---------------------------------------------------------------------------
# O6: error metrics (whole-output infinity-norm and RMS, per-element with an
# RMS floor, and a per-element rounding bound)
# ---------------------------------------------------------------------------

def rel_err_inf(y: np.ndarray, y_ref: np.ndarray) -> float:
    """max |y - y_ref| / max |y_ref| over the whole output."""
    y = np.asarray(y, dtype=np.float64)
    y_ref = np.asarray(y_ref, dtype=np.float64)
    den = np.max(np.abs(y_ref))
    if den == 0.0:
        return float(np.max(np.abs(y)))
    return float(np.max(np.abs(y - y_ref)) / den)


def rel_err_rms(y: np.ndarray, y_ref: np.ndarray) -> float:
    """||y - y_ref||_2 / ||y_ref||_2 over the whole output (RMS-relative error)."""
    y = np.asarray(y, dtype=np.float64)
    y_ref = np.asarray(y_ref, dtype=np.float64)
    den = np.sqrt(np.mean(y_ref * y_ref))
    num = np.sqrt(np.mean((y - y_ref) ** 2))
    return float(num if den == 0.0 else num / den)


def rel_err_elem(y: np.ndarray, y_ref: np.ndarray, floor: float = 1e-3) -> float:
    """max_i |y_i - y_ref_i| / max(|y_ref_i|, floor * rms(y_ref)): the worst
    per-element relative error, each element judged against its own magnitude
    but never against less than ``floor`` times the output's RMS."""
    y = np.asarray(y, dtype=np.float64)
    y_ref = np.asarray(y_ref, dtype=np.float64)
    rms = np.sqrt(np.mean(y_ref * y_ref))
    den = np.maximum(np.abs(y_ref), floor * rms)
    den = np.where(den == 0.0, 1.0, den)
    return float(np.max(np.abs(y - y_ref) / den))


def abs_inputs(spec, inputs) -> dict:
    """The same layer with every codebook value, scale and activation replaced
    by its magnitude.  Its forward is A[n, i] = sum_k |x[n, k]| |W[i, k]| with
    |W[i, k]| taken as s_i * sum_m |C[m, b, t]| (never smaller than |W|): the
    quantity that bounds every rounding error of a computed product."""
    cb = np.asarray(inputs["codebooks"])
    if spec.codebook_dtype == "bf16":
        cb_abs = (cb.astype(np.uint16) & np.uint16(0x7FFF)).astype(np.uint16)
    else:
        cb_abs = np.abs(cb)
    x = np.asarray(inputs["x"])
    x_abs = (x.astype(np.uint16) & np.uint16(0x7FFF)).astype(np.uint16) if spec.x_dtype == "bf16" else np.abs(x)
    xs = inputs.get("x_scales")
    return {"codebooks": cb_abs, "codes": inputs["codes"], "scales": np.abs(np.asarray(inputs["scales"])),
            "x": x_abs, "x_scales": None if xs is None else np.abs(np.asarray(xs))}


_UNIT = {"f16": 2.0 ** -11, "bf16": 2.0 ** -8, "f32": 2.0 ** -24}


def rounding_bound(spec, y_ref: np.ndarray, a_ref: np.ndarray, path: str) -> np.ndarray:
    """Per-element bound on |y - y_ref| for a correctly rounded computation.

    ``y_ref`` is the exact output and ``a_ref`` the forward of
    ``abs_inputs`` at the same positions.  A computed output can differ from
    the exact one only by rounding:
    * the decoded weight (path "decode"): M codewords summed with at most M-1
      roundings, times the scale, rounded once to the tile dtype, so
      |w_hat - w| <= M u_tile (1 + eps) s_i sum_m |C_m|;
    * the products and the fp32 sums over K (and, on the table path, over the
      g values of a table entry and the G M gathered entries), the scale and
      the int8 activation scale: an fp32 sum of n terms errs by at most
      gamma_n = n 2^-24 / (1 - n 2^-24) times the sum of their magnitudes;
    * the output rounding u_out |y|.
    Hence |y - y_ref| <= u_out |y_ref| + (1 + u_out) (M u_tile + gamma_n) a_ref
    (with a 1% margin on the second term), for every element.  fp16 and bf16
    activations and their products with fp16 weights are exact in fp32.
    """
    u_out = _UNIT[spec.y_dtype]
    u_tile = _UNIT[spec.tile_dtype] if path == "decode" else 0.0
    n = spec.K + spec.G * spec.M + spec.g + spec.M + 8
    e32 = 2.0 ** -24
    gamma = n * e32 / (1.0 - n * e32)
    a = np.asarray(a_ref, dtype=np.float64)
    return u_out * np.abs(np.asarray(y_ref, dtype=np.float64)) + (1.0 + u_out) * 1.01 * (spec.M * u_tile + gamma) * a


# ---------------------------------------------------------------------------
# FLOP counts of the appendix (eq. (8) and eq. (13))
# ---------------------------------------------------------------------------

def dense_conv_flops(C_out: int, C_in: int, h: int, w: int, h1: int, w1: int) -> int:
    """Dense convolution: 2 FLOP per multiply-accumulate (appendix, eq. (8))."""
    return 2 * C_out * C_in * h * w * h1 * w1


def lut_conv_flops(M: int, k: int, C_in: int, C_out: int, h: int, w: int, h1: int, w1: int) -> int:
    """LUT route of the appendix (eq. (13)), one group per (input, output) channel filter.

    Multiplications M*2^k*C_in*h*w*h1*w1 and additions M*2^k*C_in*h*w*(h1*w1-1)
    to convolve every input channel with every codeword, plus
    M*C_out*C_in*h*w additions to sum the code-indexed maps.
    """
    mults = M * (1 << k) * C_in * h * w * h1 * w1
    adds_lut = M * (1 << k) * C_in * h * w * (h1 * w1 - 1)
    adds_gather = M * C_out * C_in * h * w
    return mults + adds_lut + adds_gather


def lut_breakpoint_cout(M: int, k: int, h1w1: int) -> float:
    """Smallest C_out (real-valued) at which eq. (13) is below the dense count.

    Setting the two counts equal per (C_in, h, w):
    M 2^k (2 h1w1 - 1) + M C_out = 2 C_out h1w1, hence
    C_out = M 2^k (2 h1w1 - 1) / (2 h1w1 - M).  For a 3x3 kernel this is
    17 M 2^k / (18 - M); the closed form printed after eq. (13),
    9 (2^k - 1) M / (18 - M), does not follow from the count, and this
    function implements the count.
    """
    return M * (1 << k) * (2 * h1w1 - 1) / (2 * h1w1 - M)


# ---------------------------------------------------------------------------
# O7: codebook gradient (the continuous step of PV-Tuning, Sec. 3.2)
# ---------------------------------------------------------------------------
#
# Knowledge distillation (Sec. 3.2) tunes the codebooks of every quantized
# layer by gradient descent while the codes stay fixed between discrete
# updates; the limitations paragraph of Sec. 5 names this optimizer's cost.
# With the loss gradient dY at a layer's output, the chain rule through
# Y = X W^T gives dW = dY^T X, and through eq. (4) (with the per-row scale)
# every weight W[i, j*g + t] depends on codebook entry C[m, k, t] exactly
# when b[i, j, m] = k, with derivative s[i].  Hence
#     dC[m, k, t] = sum over (i, j) with b[i, j, m] = k of s[i] * dW[i, j*g + t].

def weight_grad_linear(X: np.ndarray, dY: np.ndarray) -> np.ndarray:
    """dW [C_out, K] = dY^T X for a linear layer (X [N, K], dY [N, C_out]), fp64."""
    return np.asarray(dY, dtype=np.float64).T @ np.asarray(X, dtype=np.float64)


def weight_grad_conv(x: np.ndarray, dy: np.ndarray, kh: int, kw: int, stride: int, pad: int) -> np.ndarray:
    """dW [C_out, C*kh*kw] of an im2col convolution (Sec. 3.1.1), fp64.

    ``x`` is the NCHW input and ``dy`` the NCHW output gradient; tokens are
    (image, output row, output column) exactly as in the forward.
    """
    cols = im2col(x, kh, kw, stride, pad)                        # [N, K]
    dy = np.asarray(dy, dtype=np.float64)
    n, C_out, OH, OW = dy.shape
    dY = dy.transpose(0, 2, 3, 1).reshape(n * OH * OW, C_out)     # token-major
    if dY.shape[0] != cols.shape[0]:
        raise ValueError("output gradient does not match the convolution geometry")
    return dY.T @ cols


def codebook_grad_from_weight_grad(dW: np.ndarray, codes: np.ndarray, scales: np.ndarray,
                                   g: int, n_entries: int) -> np.ndarray:
    """dC [M, n_entries, g] from dW [C_out, K] by the chain rule through eq. (4).

    Each (row i, group j, codebook m) adds s[i] * dW[i, j*g : (j+1)*g] to row
    b[i, j, m] of codebook m's gradient; ``np.add.at`` is the unbuffered
    scatter-add, so repeated codes accumulate.
    """
    dW = np.asarray(dW, dtype=np.float64)
    C_out, G, M = codes.shape
    if dW.shape != (C_out, G * g):
        raise ValueError("weight gradient shape does not match the codes")
    contrib = np.asarray(scales, dtype=np.float64)[:, None, None] * dW.reshape(C_out, G, g)
    dC = np.zeros((M, n_entries, g), dtype=np.float64)
    idx = codes.astype(np.int64)
    for m in range(M):
        np.add.at(dC[m], idx[:, :, m].reshape(-1), contrib.reshape(C_out * G, g))
    return dC


def codebook_grad(spec, inputs, dy: np.ndarray, x_dtype: str = None, dy_dtype: str = "f64") -> np.ndarray:
    """Gradient of the loss with respect to every codebook entry, [M, 2**B, g] fp64.

    ``inputs`` holds codes, scales and the layer input ``x`` (stored in
    ``x_dtype``, default the layer's); ``dy`` is the output gradient in the
    layer's output layout ([N, C_out] or NCHW), stored in ``dy_dtype``.
    """
    xd = spec.x_dtype if x_dtype is None else x_dtype
    X = activations_f64(inputs["x"], xd, inputs.get("x_scales"))
    dY = np.asarray(dy, dtype=np.float64) if dy_dtype == "f64" else to_f64(dy, dy_dtype)
    if spec.conv is None:
        dW = weight_grad_linear(X, dY)
    else:
        c = spec.conv
        dW = weight_grad_conv(X, dY, c.kh, c.kw, c.stride, c.pad)
    return codebook_grad_from_weight_grad(dW, inputs["codes"], inputs["scales"], spec.g, 1 << spec.B)


def codebook_grad_entries(spec, inputs, dy: np.ndarray, entries: Sequence[Sequence[int]],
                          x_dtype: str = None, dy_dtype: str = "f64") -> np.ndarray:
    """Rows dC[m, k, :] for the listed (m, k) pairs only, [len(entries), g] fp64.

    Same definition as ``codebook_grad``, evaluated one entry at a time: the
    (row, group) pairs with b[i, j, m] = k are found by a scan of the codes,
    and only their columns of dW = dY^T X are formed (tokens as im2col rows
    for a convolution), so layers too large for the full oracle stay cheap.
    """
    xd = spec.x_dtype if x_dtype is None else x_dtype
    X = activations_f64(inputs["x"], xd, inputs.get("x_scales"))
    dY = np.asarray(dy, dtype=np.float64) if dy_dtype == "f64" else to_f64(dy, dy_dtype)
    codes = inputs["codes"]
    s = np.asarray(inputs["scales"], dtype=np.float64)
    g = spec.g
    if spec.conv is not None:
        c = spec.conv
        n, C_out, OH, OW = dY.shape
        dY = dY.transpose(0, 2, 3, 1).reshape(n * OH * OW, C_out)
        _, C, H, Wd = X.shape
        xp = np.zeros((n, C, H + 2 * c.pad, Wd + 2 * c.pad), dtype=np.float64)
        xp[:, :, c.pad:c.pad + H, c.pad:c.pad + Wd] = X
    out = np.zeros((len(entries), g), dtype=np.float64)
    for e, (m, k) in enumerate(entries):
        rows, groups = np.nonzero(codes[:, :, m].astype(np.int64) == k)
        for i, j in zip(rows, groups):
            if spec.conv is None:
                cols = X[:, j * g:(j + 1) * g]
            else:
                cols = _im2col_columns(xp, c.kh, c.kw, c.stride, OH, OW, range(j * g, (j + 1) * g))
            out[e] += s[i] * (dY[:, i] @ cols)
    return out


def _im2col_columns(xp: np.ndarray, kh: int, kw: int, stride: int, OH: int, OW: int, ks) -> np.ndarray:
    """Columns ``ks`` of im2col (Sec. 3.1.1 ordering) of the zero-padded input
    ``xp``, [n*OH*OW, len(ks)], without forming the rest."""
    cols = []
    for k in ks:
        ch, rs = divmod(k, kh * kw)
        r, q = divmod(rs, kw)
        patch = xp[:, ch, r:r + stride * (OH - 1) + 1:stride, q:q + stride * (OW - 1) + 1:stride]
        cols.append(patch.reshape(-1))
    return np.stack(cols, axis=1)
