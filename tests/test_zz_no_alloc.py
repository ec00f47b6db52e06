"""The allocation-free forward (aq_layer_forward_static) against aq_layer_forward.

Same layer, same inputs: the two entry points take the same route and plan,
so their outputs must be identical bit for bit (stronger than the oracle
tolerance, which both meet; the oracle comparison is made too).  Two calls in
a row per layer, the second with a smaller input, exercise the shared static
scratch being reused with other sizes; a layer whose scratch would not fit is
refused before anything is launched.
"""
import numpy as np
import pytest
import torch

import oracle as O
from workloads import ConvGeom, LayerSpec, generate

pytestmark = pytest.mark.gpu

CASES = [
    # (spec, options, smaller n for the second call)
    (LayerSpec(name="st_tiny_f32", C_out=256, K=256, g=8, M=2, B=8, n=64, codebook_dtype="f32", x_dtype="f32",
               y_dtype="f32", tile_dtype="f32", codebook_std=0.1), {}, 17),
    (LayerSpec(name="st_lut", C_out=300, K=4096, g=8, M=2, B=8, n=40), {"lut_max_tokens": 64}, 3),
    (LayerSpec(name="st_lut_one", C_out=300, K=4096, g=8, M=4, B=8, n=40),
     {"lut_max_tokens": 64, "table_one_launch": 1}, 5),
    (LayerSpec(name="st_conv_inloop", C_out=192, K=192 * 9, g=8, M=2, B=8, n=2, conv=ConvGeom(192, 3, 3, 1, 1, 32, 32)),
     {}, 1),
    (LayerSpec(name="st_conv_split", C_out=192, K=256 * 9, g=8, M=2, B=8, n=8, conv=ConvGeom(256, 3, 3, 1, 1, 8, 8)),
     {}, 3),
    (LayerSpec(name="st_conv_rec_split", C_out=130, K=256 * 9, g=8, M=4, B=8, n=6, conv=ConvGeom(256, 3, 3, 1, 1, 8, 8)),
     {"weights": 2, "split_k": 2}, 2),
    (LayerSpec(name="st_lin_rec", C_out=1728, K=576, g=8, M=4, B=8, n=2048, x_dtype="i8"), {"weights": 2}, 700),
    (LayerSpec(name="st_dense", C_out=200, K=32 * 9, g=8, M=2, B=8, n=3, conv=ConvGeom(32, 3, 3, 1, 1, 24, 16)),
     {"weights": 2, "record_product": 2}, 1),
    (LayerSpec(name="st_kaq", C_out=96, K=32 * 9, g=9, M=2, B=8, n=2, conv=ConvGeom(32, 3, 3, 1, 1, 16, 16)), {}, 1),
    # the wave-split convolution kernel: one wave per reduction (3x3), two waves per reduction (1x1)
    (LayerSpec(name="st_ws_conv3", C_out=192, K=64 * 9, g=8, M=2, B=8, n=3, conv=ConvGeom(64, 3, 3, 1, 1, 16, 16)),
     {"weights": 2, "record_product": 3}, 1),
    (LayerSpec(name="st_ws2_conv1", C_out=128, K=128, g=8, M=2, B=8, n=4, conv=ConvGeom(128, 1, 1, 1, 0, 16, 16)),
     {"weights": 2, "record_product": 3, "fused_tile": "64x128"}, 2),
]


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.mark.parametrize("spec,opts,n2", CASES, ids=[c[0].name for c in CASES])
def test_static_forward_matches_forward(spec, opts, n2):
    import paper_2506_05960_amd as P
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need an MI355X; none is visible")
    inp = generate(spec, 808)
    layer = P.AQLayer(spec, inp)
    for k, v in opts.items():
        layer.set_option(k, v)
    print(f"static {spec.name}: {layer.describe(spec.n)}", flush=True)
    for n in (spec.n, n2):
        x = _dev(inp["x"][:n])
        xs = None if inp["x_scales"] is None else _dev(inp["x_scales"][:layer.tokens(n)])
        y_ref = layer.forward(x, xs)
        y_st = layer.forward(x, xs, static=True)
        torch.cuda.synchronize()
        assert torch.equal(y_st, y_ref), f"{spec.name} n={n}: the static forward differs from the forward"
        sub = dict(inp)
        sub["x"] = inp["x"][:n]
        if inp["x_scales"] is not None:
            sub["x_scales"] = inp["x_scales"][:layer.tokens(n)]
        tol = 1e-5 if spec.tile_dtype == "f32" and spec.y_dtype == "f32" else 2e-3
        assert O.rel_err_inf(y_st.float().cpu().numpy(), O.forward(spec.with_n(n), sub)) <= tol
    layer.close()


def test_static_forward_in_a_graph_and_repeated():
    import paper_2506_05960_amd as P
    spec = CASES[4][0]
    inp = generate(spec, 809)
    layer = P.AQLayer(spec, inp)
    x = _dev(inp["x"])
    ref = layer.forward(x).clone()
    y = torch.zeros_like(ref)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            layer.forward(x, out=y, static=True)
    torch.cuda.current_stream().wait_stream(s)
    for rep in range(3):
        y.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, ref), rep
        assert torch.equal(layer.forward(x, static=True), ref)
    layer.close()


def test_static_forward_refuses_scratch_beyond_the_array():
    import paper_2506_05960_amd as P
    # pre-decoded records of 4096 x 8192 fp16 weights: 64 MiB, above the static array's data area
    spec = LayerSpec(name="st_big", C_out=4096, K=8192, g=8, M=2, B=8, n=64)
    inp = generate(spec, 810)
    layer = P.AQLayer(spec, inp)
    layer.set_option("weights", 2)
    x = _dev(inp["x"])
    y = torch.full((64, 4096), 7.0, dtype=torch.float16, device="cuda")
    with pytest.raises(P.AQError, match="AQ_ERR_UNSUPPORTED"):
        layer.forward(x, out=y, static=True)
    torch.cuda.synchronize()
    assert bool((y == 7.0).all())            # nothing was launched
    layer.close()
