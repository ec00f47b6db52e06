"""GPU parity along the chained U-Net pass (batch 8, W2).

The pass is built as the benchmark builds it: a residual block's skip
convolution reads the block's input buffer, as the block's first 3x3
convolution does (``workloads.branch_inputs``); any other layer i reads layer
i-1's output buffer where the element counts allow
(``workloads.chain_sources``), else a seeded buffer of its own; codebooks
have the unit-scale standard deviation.  After one eager pass every layer's
sampled outputs are compared with the oracle evaluated on that layer's actual
GPU input, and replays of the whole pass from a HIP graph (in layer order on
one stream, and as the benchmark times it: the batched record decodes first,
the skips on a second stream) must reproduce every output bit for bit.
"""
import sys

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from parity_checks import check_against_oracle, edge_samples, sampled_outputs

pytestmark = pytest.mark.gpu

LAYERS = W.sweep_layers(full=False)


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def chain():
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need an MI355X; none is visible")
    import paper_2506_05960_amd as P
    P.load_library()
    src = W.chain_sources(LAYERS, batch=8)
    branch = W.branch_inputs(LAYERS)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(W.SEED_BASE + 4)
    built, prev = [], None
    for i, lay in enumerate(LAYERS):
        spec = W.sweep_spec(lay, 2, batch=8, codebook_std="chain")
        wts = W.generate(spec.with_n(1), W.SEED_BASE + 100 + i)
        layer = P.AQLayer(spec, wts, max_tokens=spec.tokens)
        xs = layer.in_shape(spec.n)
        if branch[i] is not None:
            x = built[branch[i]][3]
            assert tuple(x.shape) == tuple(xs)
        elif src[i] is not None:
            x = prev.view(xs)
        else:
            x = torch.randn(xs, generator=gen, device="cuda", dtype=torch.float32).to(torch.float16)
        y = torch.empty(layer.out_shape(spec.n), dtype=torch.float16, device="cuda")
        built.append((spec, wts, layer, x, y))
        prev = y
    _say(f"chained pass: {len(LAYERS)} layers, {sum(s is not None for s in src)} chained")
    for _, _, layer, x, y in built:
        layer.forward(x, None, out=y)
    torch.cuda.synchronize()
    snap = [(x.cpu().numpy(), y.float().cpu().numpy().astype(np.float64), layer.choose_path(spec.tokens))
            for spec, _, layer, x, y in built]
    yield built, snap, src, branch
    for _, _, layer, _, _ in built:
        layer.close()


@pytest.mark.parametrize("i", range(len(LAYERS)), ids=[l.name for l in LAYERS])
def test_chained_layer_matches_oracle_on_its_gpu_input(chain, i):
    built, snap, src, branch = chain
    spec, wts, _, _, _ = built[i]
    x_host, y_host, path = snap[i]
    inp = dict(wts)
    inp["x"] = x_host
    inp["x_scales"] = None
    rms = float(np.sqrt(np.mean(y_host ** 2)))
    where = "block input" if branch[i] is not None else "prev" if src[i] is not None else "own"
    _say(f"chain {i} {spec.name} input={where} out_rms={rms:.3f}")
    assert 0.2 < rms < 5.0            # unit scale along the chain: no blow-up, no collapse
    tok, ch = edge_samples(spec, np.random.default_rng(i))
    check_against_oracle(spec, inp, sampled_outputs(spec, y_host, tok, ch), tok, ch, path, 2e-3)


def test_chained_pass_graph_replay_is_bitwise_identical(chain):
    built, snap, _, _ = chain
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            for _, _, layer, x, y in built:
                layer.forward(x, None, out=y)
    torch.cuda.current_stream().wait_stream(s)
    for rep in range(3):
        for _, _, _, _, y in built:
            y.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for j, (_, _, _, _, y) in enumerate(built):
            assert np.array_equal(y.float().cpu().numpy().astype(np.float64), snap[j][1]), (rep, j)


def test_two_stream_pass_with_batched_decodes_is_bitwise_identical(chain):
    """The benchmark's schedule: every layer's record decodes batched first (aq_layers_prepare), then the pass
    with each residual skip convolution on a second stream beside its block's 3x3 convolutions; captured in one
    graph and replayed three times, with an eager forward in between, against the eager one-stream pass."""
    import bench
    import paper_2506_05960_amd as P
    built, snap, _, branch = chain
    layers = [b[2] for b in built]
    ns = [b[0].n for b in built]
    fns = [(lambda layer=layer, x=x, y=y: layer.forward(x, None, out=y)) for _, _, layer, x, y in built]
    main = torch.cuda.current_stream()
    s = torch.cuda.Stream()
    side = torch.cuda.Stream()
    s.wait_stream(main)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            bench.run_pass_branches(torch, fns, branch, side, first=lambda: P.AQLayer.prepare_all(layers, ns))
    main.wait_stream(s)
    for rep in range(3):
        for _, _, _, _, y in built:
            y.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for j, (_, _, _, _, y) in enumerate(built):
            assert np.array_equal(y.float().cpu().numpy().astype(np.float64), snap[j][1]), (rep, j)
        j = 11 * rep % len(built)
        fns[j]()                                   # an eager forward between replays (decodes its own records)
        torch.cuda.synchronize()
        assert np.array_equal(built[j][4].float().cpu().numpy().astype(np.float64), snap[j][1]), (rep, j)
