"""Layer specifications and seeded generators for synthetic AQ layers.

Storage conventions (these are the conventions of the library boundary too):

* codebooks ``[M][2**B][g]`` in the codebook dtype (fp32, fp16, or bf16 kept as
  ``uint16`` bit patterns, since numpy has no bfloat16);
* codes ``[C_out][K // g][M]``: ``uint8`` when ``B <= 8``, else ``uint16``;
* scales ``[C_out]`` fp32, one per output channel;
* linear activations ``[N][K]`` row-major; convolution activations NCHW
  ``[n][C_in][H][W]``;
* int8 activations carry a per-token fp32 scale ``x_scales[N]``.

Workload shapes follow the LDM-4 ImageNet-256 U-Net that the paper evaluates
(Sec. 4, Table 3): model width 192 with channel multipliers (1, 2, 3, 5) at
latent resolutions 64/32/16/8.  No dataset item or trained weight is used:
every value is drawn from a seeded numpy PCG64 generator, in the fixed order
codebooks, codes, scales, activations, activation scales.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np

SEED_BASE = 2506_05960

_DTYPES = ("f32", "f16", "bf16", "i8")


@dataclass(frozen=True)
class ConvGeom:
    """Geometry of a 2-D convolution lowered to a matmul by im2col (Sec. 3.1.1)."""

    cin: int
    kh: int
    kw: int
    stride: int
    pad: int
    H: int
    W: int

    @property
    def OH(self) -> int:
        return (self.H + 2 * self.pad - self.kh) // self.stride + 1

    @property
    def OW(self) -> int:
        return (self.W + 2 * self.pad - self.kw) // self.stride + 1

    @property
    def K(self) -> int:
        return self.cin * self.kh * self.kw


@dataclass(frozen=True)
class LayerSpec:
    """One AQ layer: format (g, M, B), dtypes, geometry and token count.

    ``n`` is the number of tokens for a linear layer and the batch size for a
    convolution (tokens = n * OH * OW).
    """

    name: str
    C_out: int
    K: int
    g: int
    M: int
    B: int
    n: int
    codebook_dtype: str = "f16"
    x_dtype: str = "f16"
    y_dtype: str = "f16"
    tile_dtype: str = "f16"
    codebook_std: float = 0.05
    x_std: float = 1.0
    conv: Optional[ConvGeom] = None
    note: str = ""

    def __post_init__(self):
        if self.K % self.g:
            raise ValueError(f"{self.name}: K={self.K} not divisible by g={self.g}")
        if self.conv is not None and self.conv.K != self.K:
            raise ValueError(f"{self.name}: conv K mismatch")
        for d in (self.codebook_dtype, self.x_dtype, self.y_dtype, self.tile_dtype):
            if d not in _DTYPES:
                raise ValueError(d)

    @property
    def G(self) -> int:
        return self.K // self.g

    @property
    def tokens(self) -> int:
        if self.conv is None:
            return self.n
        return self.n * self.conv.OH * self.conv.OW

    @property
    def code_dtype(self):
        return np.uint8 if self.B <= 8 else np.uint16

    @property
    def dense_flops(self) -> int:
        """Dense-equivalent FLOPs of one forward: 2 per multiply-accumulate."""
        return 2 * self.tokens * self.K * self.C_out

    def with_n(self, n: int) -> "LayerSpec":
        return dataclasses.replace(self, n=n)

    def to_dict(self) -> dict:
        d = dataclasses.asdict(self)
        return d


def _round_bf16_bits(x64: np.ndarray) -> np.ndarray:
    """fp64 -> bf16 (round to nearest even through torch's cast), as uint16 bits."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(x64, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def _cast(x64: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return x64.astype(np.float32)
    if dtype == "f16":
        return x64.astype(np.float16)
    if dtype == "bf16":
        return _round_bf16_bits(x64)
    raise ValueError(dtype)


def generate(spec: LayerSpec, seed: int) -> Dict[str, np.ndarray]:
    """Draw every input of ``spec`` from ``default_rng(seed)``.

    Returns a dict with ``codebooks``, ``codes``, ``scales``, ``x`` and
    ``x_scales`` (``None`` unless ``x_dtype == 'i8'``).
    """
    rng = np.random.default_rng(seed)
    M, B, g = spec.M, spec.B, spec.g
    cb = rng.normal(0.0, spec.codebook_std, size=(M, 1 << B, g))
    codebooks = _cast(cb, spec.codebook_dtype)
    codes = rng.integers(0, 1 << B, size=(spec.C_out, spec.G, M), dtype=np.int64).astype(spec.code_dtype)
    scales = rng.uniform(0.5, 1.5, size=spec.C_out).astype(np.float32)
    if spec.conv is None:
        xshape = (spec.n, spec.K)
    else:
        c = spec.conv
        xshape = (spec.n, c.cin, c.H, c.W)
    x_scales = None
    if spec.x_dtype == "i8":
        q = np.clip(np.rint(rng.normal(0.0, 30.0, size=xshape)), -127, 127)
        x = q.astype(np.int8)
        ntok = xshape[0]
        x_scales = (rng.uniform(0.5, 1.5, size=ntok) / 127.0).astype(np.float32)
    else:
        x = _cast(rng.normal(0.0, spec.x_std, size=xshape), spec.x_dtype)
    return {"codebooks": codebooks, "codes": codes, "scales": scales, "x": x, "x_scales": x_scales}


def generate_grad_inputs(spec: LayerSpec, seed: int, dtype: str = "f16") -> Dict[str, np.ndarray]:
    """Layer input ``x`` and output gradient ``dy`` for the codebook gradient.

    Both are drawn from ``default_rng(seed)`` as N(0, x_std) and N(0, 1) in
    ``dtype`` (fp16, or bf16 as uint16 bits), in the forward's layouts:
    [n, K] and [n, C_out] for a linear layer, NCHW for a convolution.
    """
    rng = np.random.default_rng(seed)
    if spec.conv is None:
        xshape, yshape = (spec.n, spec.K), (spec.n, spec.C_out)
    else:
        c = spec.conv
        xshape, yshape = (spec.n, c.cin, c.H, c.W), (spec.n, spec.C_out, c.OH, c.OW)
    x = _cast(rng.normal(0.0, spec.x_std, size=xshape), dtype)
    dy = _cast(rng.normal(0.0, 1.0, size=yshape), dtype)
    return {"x": x, "dy": dy}


# ---------------------------------------------------------------------------
# The four single-layer workloads plus the LDM-4-shaped sweep.
# ---------------------------------------------------------------------------

def _tiny() -> LayerSpec:
    return LayerSpec(
        name="tiny_linear_64x256_to_256_g8_M2_B8_f32",
        C_out=256, K=256, g=8, M=2, B=8, n=64,
        codebook_dtype="f32", x_dtype="f32", y_dtype="f32", tile_dtype="f32",
        codebook_std=0.1,
    )


def _conv64() -> LayerSpec:
    geom = ConvGeom(cin=192, kh=3, kw=3, stride=1, pad=1, H=64, W=64)
    return LayerSpec(
        name="conv3x3_64x64_b2_192to192_g8_M2_B8_f16",
        C_out=192, K=geom.K, g=8, M=2, B=8, n=2, conv=geom,
    )


def _qkv16() -> LayerSpec:
    return LayerSpec(
        name="qkv_16x16_8192tok_576to1728_g8_M4_B8_a8",
        C_out=1728, K=576, g=8, M=4, B=8, n=8192, x_dtype="i8",
    )


def _conv8() -> LayerSpec:
    geom = ConvGeom(cin=960, kh=3, kw=3, stride=1, pad=1, H=8, W=8)
    return LayerSpec(
        name="conv3x3_8x8_b64_960to960_g8_M1_B16_f16",
        C_out=960, K=geom.K, g=8, M=1, B=16, n=64, conv=geom,
    )


CONFIGS: Dict[str, LayerSpec] = {
    "tiny": _tiny(),
    "conv64": _conv64(),
    "qkv16": _qkv16(),
    "conv8": _conv8(),
}

_CONFIG_INDEX = {"tiny": 0, "conv64": 1, "qkv16": 2, "conv8": 3, "sweep": 4}


def config_spec(name: str) -> LayerSpec:
    return CONFIGS[name]


def config_inputs(name: str) -> Dict[str, np.ndarray]:
    return generate(CONFIGS[name], SEED_BASE + _CONFIG_INDEX[name])


# ---------------------------------------------------------------------------
# LDM-4-shaped U-Net layer list (synthetic stand-in for the paper's workload).
# ---------------------------------------------------------------------------

@dataclass(frozen=True)
class SweepLayer:
    name: str
    kind: str          # "conv3x3", "conv1x1", "linear"
    cin: int           # K for linear
    cout: int
    res: int           # input spatial resolution (conv) / token grid side (linear)
    stride: int = 1
    tokens_per_image: Optional[int] = None  # linear layers; default res*res
    role: str = ""

    def macs(self, batch: int) -> int:
        if self.kind == "linear":
            t = self.tokens_per_image if self.tokens_per_image is not None else self.res * self.res
            return batch * t * self.cin * self.cout
        k = 3 if self.kind == "conv3x3" else 1
        o = self.res // self.stride
        return batch * o * o * self.cin * k * k * self.cout


def sweep_layers(full: bool = False) -> List[SweepLayer]:
    """Quantized layers of an LDM-4-style U-Net (width 192, mult 1/2/3/5).

    ``full=False`` keeps the "strict" reading (3x3/1x1 convs, fused qkv and
    attention-output linears); ``full=True`` adds the remaining transformer
    linears, including the cross-attention key/value projection, which runs on
    one context token per image.  conv_in/conv_out and the time-embedding
    linears stay unquantized in the paper and are excluded.
    """
    ch = [192, 384, 576, 960]
    res = [64, 32, 16, 8]
    out: List[SweepLayer] = []

    def resblock(tag, cin, cout, r):
        out.append(SweepLayer(f"{tag}.conv1", "conv3x3", cin, cout, r, role="res"))
        out.append(SweepLayer(f"{tag}.conv2", "conv3x3", cout, cout, r, role="res"))
        if cin != cout:
            out.append(SweepLayer(f"{tag}.skip", "conv1x1", cin, cout, r, role="res_skip"))

    def transformer(tag, c, r):
        if full:
            out.append(SweepLayer(f"{tag}.proj_in", "linear", c, c, r, role="attn"))
        out.append(SweepLayer(f"{tag}.attn1.qkv", "linear", c, 3 * c, r, role="attn"))
        out.append(SweepLayer(f"{tag}.attn1.out", "linear", c, c, r, role="attn"))
        if full:
            out.append(SweepLayer(f"{tag}.attn2.q", "linear", c, c, r, role="attn"))
            out.append(SweepLayer(f"{tag}.attn2.kv", "linear", 512, 2 * c, r,
                                  tokens_per_image=1, role="attn_ctx"))
            out.append(SweepLayer(f"{tag}.attn2.out", "linear", c, c, r, role="attn"))
            out.append(SweepLayer(f"{tag}.ff.in", "linear", c, 8 * c, r, role="ff"))
            out.append(SweepLayer(f"{tag}.ff.out", "linear", 4 * c, c, r, role="ff"))
            out.append(SweepLayer(f"{tag}.proj_out", "linear", c, c, r, role="attn"))

    skips = [ch[0]]  # conv_in output
    cur = ch[0]
    for lvl in range(4):
        for b in range(2):
            resblock(f"down{lvl}.{b}", cur, ch[lvl], res[lvl])
            cur = ch[lvl]
            if lvl >= 1:
                transformer(f"down{lvl}.{b}.tf", cur, res[lvl])
            skips.append(cur)
        if lvl < 3:
            out.append(SweepLayer(f"down{lvl}.downsample", "conv3x3", cur, cur, res[lvl],
                                  stride=2, role="downsample"))
            skips.append(cur)
    resblock("mid.0", cur, cur, res[3])
    transformer("mid.tf", cur, res[3])
    resblock("mid.1", cur, cur, res[3])
    for lvl in (3, 2, 1, 0):
        for b in range(3):
            s = skips.pop()
            resblock(f"up{lvl}.{b}", cur + s, ch[lvl], res[lvl])
            cur = ch[lvl]
            if lvl >= 1:
                transformer(f"up{lvl}.{b}.tf", cur, res[lvl])
        if lvl > 0:
            out.append(SweepLayer(f"up{lvl}.upsample", "conv3x3", cur, cur, res[lvl - 1],
                                  role="upsample"))
    assert not skips
    return out


def unet_attention_macs(batch: int) -> int:
    """MACs of the non-weight attention matmuls (Q.K^T and A.V) of the same U-Net.

    Self-attention over T = R*R tokens costs 2*T*T*C per image; cross-attention
    over one context token costs 2*T*C.  Used only to check the layer list
    against the paper's full-precision FLOP total.
    """
    ch = [192, 384, 576, 960]
    res = [64, 32, 16, 8]
    n_tf = {1: 5, 2: 5, 3: 6}  # 2 encoder + 3 decoder (+1 middle at level 3)
    tot = 0
    for lvl, cnt in n_tf.items():
        t = res[lvl] ** 2
        tot += cnt * (2 * t * t * ch[lvl] + 2 * t * ch[lvl])
    return batch * tot


def unet_unquantized_conv_macs(batch: int, latent_ch: int = 3) -> int:
    """conv_in (latent->192) and conv_out (192->latent), 3x3 at 64x64."""
    return batch * 2 * 64 * 64 * 9 * latent_ch * 192


def sweep_spec(layer: SweepLayer, M: int, batch: int = 8, B: int = 8, g: int = 8,
               codebook_std: Optional[float] = None) -> LayerSpec:
    """AQ layer spec of one sweep layer (fp16 activations, fp16 codebooks).

    ``codebook_std`` defaults to 0.05; ``"chain"`` selects the unit-scale
    value of ``chain_codebook_std``."""
    variant = f"W{M * B // g}"
    if layer.kind == "linear":
        t = layer.tokens_per_image if layer.tokens_per_image is not None else layer.res * layer.res
        K = layer.cin
        geom = None
        n = batch * t
    else:
        k = 3 if layer.kind == "conv3x3" else 1
        geom = ConvGeom(cin=layer.cin, kh=k, kw=k, stride=layer.stride, pad=(k - 1) // 2,
                        H=layer.res, W=layer.res)
        K = geom.K
        n = batch
    std = 0.05 if codebook_std is None else (chain_codebook_std(M, K) if codebook_std == "chain" else codebook_std)
    return LayerSpec(name=f"{layer.name}.{variant}", C_out=layer.cout, K=K, g=g, M=M, B=B, n=n, conv=geom,
                     note=layer.role, codebook_std=float(std))


def sweep_io_elems(layer: SweepLayer, batch: int):
    """(input elements, output elements) of one sweep layer at ``batch``."""
    if layer.kind == "linear":
        t = batch * (layer.tokens_per_image if layer.tokens_per_image is not None else layer.res * layer.res)
        return t * layer.cin, t * layer.cout
    o = layer.res // layer.stride
    return batch * layer.cin * layer.res * layer.res, batch * layer.cout * o * o


def chain_sources(layers: List[SweepLayer], batch: int = 8) -> List[Optional[int]]:
    """For a chained pass over ``layers``: entry i is i - 1 when the previous
    layer's output buffer can serve as layer i's input (same element count:
    a convolution output [n, C, R, R] is read as the [n*R*R, C] tokens of a
    following linear layer and back), else None (layer i reads a buffer of
    its own).  The U-Net's glue between layers (normalisation, attention,
    up-sampling, skip concatenation) is not part of the pass."""
    src: List[Optional[int]] = []
    for i, lay in enumerate(layers):
        if i > 0 and sweep_io_elems(layers[i - 1], batch)[1] == sweep_io_elems(lay, batch)[0]:
            src.append(i - 1)
        else:
            src.append(None)
    return src


def branch_inputs(layers: List[SweepLayer]) -> List[Optional[int]]:
    """For a chained pass over ``layers``: entry i is the index of the earlier
    layer whose input buffer layer i reads too, else None.  A residual block's
    1x1 skip convolution reads the block's input, as the block's first 3x3
    convolution does; it depends on nothing in between, so it may run
    concurrently with the block's two 3x3 convolutions, and the layer after
    it (which reads the block's output, the sum of the two branches) waits for
    both."""
    idx = {lay.name: i for i, lay in enumerate(layers)}
    out: List[Optional[int]] = []
    for lay in layers:
        if lay.role == "res_skip":
            out.append(idx[lay.name.rsplit(".", 1)[0] + ".conv1"])
        else:
            out.append(None)
    return out


def chain_codebook_std(M: int, K: int) -> float:
    """Codebook standard deviation that keeps a chained layer's output at unit
    scale for unit-scale input: with scales U(0.5, 1.5) (mean square 13/12),
    M codewords per group and K inputs, var(y) = (13/12) K M sigma^2."""
    return 1.0 / np.sqrt(13.0 / 12.0 * M * K)


def lut_regime_specs(n_list=(1, 2, 4, 8, 16, 32, 64)) -> List[LayerSpec]:
    """Small-token-count linear layers with sweep shapes (the LUT kernel's regime)."""
    shapes = [(576, 1728), (960, 2880), (8640, 960), (17280, 960)]
    out = []
    for (K, C) in shapes:
        for M in (2, 4):
            for n in n_list:
                out.append(LayerSpec(name=f"lut_{K}to{C}_M{M}_n{n}", C_out=C, K=K, g=8, M=M, B=8, n=n))
    return out
