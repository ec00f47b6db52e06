"""Benchmark of the AQ layer forward on one MI355X.

One step = the whole hot path (dispatch, activation staging, weight decode or
table build, contraction, epilogue) over one batch of synthetic input that is
resident in HBM before timing starts.  The default workload is the
LDM-4-shaped U-Net pass at batch 8 (W2: g = 8, M = 2, B = 8): its 97
quantized layers chained, one step per pass.  ``--config conv64|qkv16|conv8|
tiny`` times one layer instead (one step per forward).  Prints ONE JSON line
with dense-equivalent TFLOP/s (2 FLOP per multiply-accumulate), the
algorithmic HBM GB/s, the roofline fraction of the dominant kernel (timed
live with HIP events around every launch) and the CPU oracle timed on this
host.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config sweep]
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_MFMA_F16_TFLOPS = 2500.0   # MI355X dense fp16/bf16 matrix-core peak
PEAK_HBM_GBS = 8000.0           # MI355X HBM3E
PEAK_F32_VALU_TFLOPS = 157.3


def _dtype_bytes(name: str) -> int:
    return {"f32": 4, "f16": 2, "bf16": 2, "i8": 1}[name]


def algorithmic_bytes(spec) -> int:
    """Bytes the layer must move at least once: codes, codebooks, scales, X, Y.

    Convolutions count the NCHW input once (implicit im2col), not the im2col
    matrix.  int8 activations add their per-token scales.
    """
    code_b = 1 if spec.B <= 8 else 2
    codes = spec.C_out * spec.G * spec.M * code_b
    cbs = spec.M * (1 << spec.B) * spec.g * _dtype_bytes(spec.codebook_dtype)
    scales = 4 * spec.C_out
    if spec.conv is None:
        x = spec.n * spec.K * _dtype_bytes(spec.x_dtype)
    else:
        c = spec.conv
        x = spec.n * c.cin * c.H * c.W * _dtype_bytes(spec.x_dtype)
    xs = 4 * spec.tokens if spec.x_dtype == "i8" else 0
    y = spec.tokens * spec.C_out * _dtype_bytes(spec.y_dtype)
    return codes + cbs + scales + x + xs + y


def kernel_source_hash() -> str:
    """SHA-256 over the HIP sources and headers that make up the library."""
    h = hashlib.sha256()
    files = sorted(glob.glob(os.path.join(ROOT, "paper_2506_05960_amd", "csrc", "*")) +
                   glob.glob(os.path.join(ROOT, "include", "*.h")))
    for f in files:
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def host_info():
    """CPU model, usable cores and the BLAS library numpy's matmul runs on."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    cores = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    blas, threads = "unknown", cores
    try:
        from threadpoolctl import threadpool_info
        info = [p for p in threadpool_info() if p.get("user_api") == "blas"]
        if info:
            blas = f"{info[0].get('internal_api')} {info[0].get('version')}"
            threads = int(info[0].get("num_threads", cores))
    except Exception:
        pass
    return {"cpu": model, "cores_available": cores, "blas": blas, "threads": threads}


def cpu_baseline(spec, inp, budget_s: float = 12.0):
    """Time the fp64 oracle on this host's cores (bounded number of repetitions)."""
    import oracle as O

    hi = host_info()
    t0 = time.perf_counter()
    O.forward(spec, inp)       # warm-up
    first = time.perf_counter() - t0
    reps = max(1, min(5, int(budget_s / max(first, 1e-3))))
    times = []
    for _ in range(reps):
        t0 = time.perf_counter()
        O.forward(spec, inp)
        times.append(time.perf_counter() - t0)
    t = statistics.median(times)
    return {
        "value": round(spec.dense_flops / t / 1e12, 6),
        "unit": "TFLOP/s",
        "cores": int(hi["threads"]),
        "kind": "oracle",
        "sample": f"whole layer ({spec.name}): fp64 dequantize + im2col + BLAS matmul, "
                  f"median of {reps} runs after 1 warm-up, {t:.3f} s per forward",
        "cpu": hi["cpu"],
        "blas": hi["blas"],
    }


def _graph_time_us(torch, fn, reps: int, trials: int = 5) -> float:
    """Median per-call time of `fn` replayed from a HIP graph of `reps` calls (HIP events)."""
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    fn()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(stream):
        with torch.cuda.graph(graph, stream=stream):
            for _ in range(reps):
                fn()
    torch.cuda.current_stream().wait_stream(stream)
    graph.replay()
    torch.cuda.synchronize()
    times = []
    for _ in range(trials):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        graph.replay()
        b.record()
        torch.cuda.synchronize()
        times.append(a.elapsed_time(b) * 1e3 / reps)
    return statistics.median(times)


PRODUCT_KERNELS = ("fused_fwd_kernel", "rec_conv_kernel", "rec_linear_kernel", "rec_gemm_kernel", "mfma_fwd_kernel",
                   "f32_fwd_kernel", "lut_fwd_kernel")


def launch_times(torch, items, replays: int = 5, graph_reps: int = 10):
    """Per-launch kernel durations of a pass of forwards, timed with HIP events.

    ``items`` is a list of (layer, fn): ``fn()`` runs the layer's forward (a
    layer may repeat).  Two measurements, both with HIP events on the launch
    stream:

    * each distinct forward alone, ``graph_reps`` times in one HIP graph: its
      duration without launch gaps (for a one-launch forward, the kernel's);
    * the launches of a forward split by timing events that the library
      records around each of them (aq_layer_set_launch_events).  The runtime
      records no events inside a captured graph, so this pass runs eagerly,
      queued twice back to back with events only in the second (the host
      queues it while the GPU runs the first, so no launch waits for the host,
      and no event is re-recorded while a record is pending).  Eager launches
      carry gaps, so these times only apportion the graph-timed forward among
      its launches.

    Returns (per-layer list of (kernel name, us)), "graph", median eager pass
    us with the events).
    """
    layouts = []
    for layer, fn in items:
        fn()
        torch.cuda.synchronize()
        n, names = layer.last_launches()
        layouts.append(names[:n])
    fwd_us = {}
    for layer, fn in items:
        if id(layer) not in fwd_us:
            fwd_us[id(layer)] = _graph_time_us(torch, fn, reps=graph_reps)
    evs = []
    for (layer, _), names in zip(items, layouts):
        e = [torch.cuda.Event(enable_timing=True) for _ in range(len(names) + 1)]
        for x in e:
            x.record()
        evs.append(e)
    torch.cuda.synchronize()
    samples = [[[] for _ in names] for names in layouts]
    pass_us = []
    for _ in range(replays):
        for layer, fn in items:
            layer.set_launch_events([])
            fn()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for (layer, fn), e in zip(items, evs):
            layer.set_launch_events(e)
            fn()
        b.record()
        for layer, _ in items:
            layer.set_launch_events([])
        torch.cuda.synchronize()
        pass_us.append(a.elapsed_time(b) * 1e3)
        for li, e in enumerate(evs):
            for k in range(len(e) - 1):
                samples[li][k].append(e[k].elapsed_time(e[k + 1]) * 1e3)
    per_layer = []
    for li, names in enumerate(layouts):
        ev = [statistics.median(samples[li][k]) for k in range(len(names))]
        tot = sum(ev) or 1.0
        g = fwd_us[id(items[li][0])]
        per_layer.append([(names[k], g * ev[k] / tot) for k in range(len(names))])
    return per_layer, "graph", statistics.median(pass_us)


def dominant_kernel(per_layer, flops):
    """Group launches by kernel; the dominant one takes the most time.  Its
    achieved rate is the dense FLOPs of the layers it computes over its
    total duration (auxiliary launches: record decoding, reductions, packing,
    carry no FLOPs of their own)."""
    tot, cnt, fl = {}, {}, {}
    for li, launches in enumerate(per_layer):
        for name, us in launches:
            tot[name] = tot.get(name, 0.0) + us
            cnt[name] = cnt.get(name, 0) + 1
            if name.startswith(PRODUCT_KERNELS):
                fl[name] = fl.get(name, 0) + flops[li]
    name = max(tot, key=tot.get)
    table = sorted(((n, tot[n], cnt[n], fl.get(n, 0)) for n in tot), key=lambda r: -r[1])
    return name, tot[name], cnt[name], fl.get(name, 0), table


def measured_traffic_kernel(workload: str, kernel: str):
    """HBM bytes per launch of ``kernel`` in ``workload`` from the committed counter summary (or None)."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as f:
            d = json.load(f)
    except (OSError, ValueError):
        return None
    ent = d.get(f"{workload}:{kernel}")
    if not ent or ent.get("source_hash") != kernel_source_hash():
        return None
    return ent.get("traffic_bytes")


def sweep_cpu_baseline(specs, seeds, budget_s: float = 25.0, stride: int = 1):
    """The fp64 oracle over the pass's layers (every ``stride``-th, in order,
    until the budget is spent: the whole pass takes about 16 s on 16 threads),
    each with its own weights and a seeded N(0, 1) input of the full batch."""
    import numpy as np

    import oracle as O
    import workloads as W

    hi = host_info()
    done, flops, t_all = [], 0, 0.0
    for i in range(0, len(specs), stride):
        spec = specs[i]
        inp = W.generate(spec, seeds[i])
        t0 = time.perf_counter()
        O.forward(spec, inp)
        t_all += time.perf_counter() - t0
        flops += spec.dense_flops
        done.append(spec.name)
        if t_all > budget_s:
            break
    return {
        "value": round(flops / t_all / 1e12, 6),
        "unit": "TFLOP/s",
        "cores": int(hi["threads"]),
        "kind": "oracle",
        "sample": f"{len(done)} of the pass's {len(specs)} layers ({'every layer' if stride == 1 else f'every {stride}th'}"
                  f", in order, {flops / 1e9:.1f} GFLOP): fp64 "
                  f"dequantize + im2col + BLAS matmul, one run each, {t_all:.2f} s",
        "cpu": hi["cpu"],
        "blas": hi["blas"],
    }


def dense_gemm_reference(torch, specs, gen):
    """Each layer of a pass as a dense fp16 GEMM through torch.matmul (hipBLASLt):
    [tokens, K] x [K, C_out] with the weights stored [C_out, K] (the faster of
    the two weight layouts there), seeded N(0, 1) operands, fp16 output, im2col
    not counted.  A comparator for what unquantized fp16 weights cost in the
    vendor library on the same shapes, not a step of the method.  Returns the
    per-layer matmul callables."""
    mx_a = max(sp.tokens * sp.K for sp in specs)
    mx_w = max(sp.K * sp.C_out for sp in specs)
    mx_y = max(sp.tokens * sp.C_out for sp in specs)
    A = torch.randn(mx_a, generator=gen, device="cuda", dtype=torch.float16)
    Wt = torch.randn(mx_w, generator=gen, device="cuda", dtype=torch.float16)
    Yd = torch.empty(mx_y, device="cuda", dtype=torch.float16)
    fns = []
    for sp in specs:
        a = A[:sp.tokens * sp.K].view(sp.tokens, sp.K)
        w = Wt[:sp.C_out * sp.K].view(sp.C_out, sp.K)
        y = Yd[:sp.tokens * sp.C_out].view(sp.tokens, sp.C_out)
        fns.append(lambda a=a, w=w, y=y: torch.matmul(a, w.t(), out=y))
    return fns


def run_pass_branches(torch, fns, branch, side, first=None):
    """Launch one U-Net pass: ``fns[i]()`` queues layer i's forward on the
    current stream.  A layer that reads an earlier layer's input
    (``branch[i] = j``: a residual block's skip convolution reads the block
    input, as its first 3x3 convolution j does) goes to the ``side`` stream as
    soon as that input is ready (just before layer j), and the next layer in
    order that is not such a branch waits for it; every other layer runs in
    order on the current stream.  ``first()`` (say, the batched record
    decodes) runs before anything else, and both streams start after it."""
    main = torch.cuda.current_stream()
    if first is not None:
        first()
    starts = {}
    for i, j in enumerate(branch):
        if j is not None:
            starts.setdefault(j, []).append(i)
    joins = []                                   # (first layer that waits, event)
    for i, fn in enumerate(fns):
        for k in starts.get(i, ()):
            side.wait_stream(main)
            with torch.cuda.stream(side):
                fns[k]()
            ev = torch.cuda.Event()
            ev.record(side)
            joins.append((k + 1, ev))
        if branch[i] is not None:
            continue
        for t, ev in [je for je in joins if je[0] <= i]:
            main.wait_event(ev)
        joins = [je for je in joins if je[0] > i]
        fn()
    for _, ev in joins:
        main.wait_event(ev)


def sweep_bench(a, torch, P, W):
    """The LDM-4-shaped U-Net pass at batch 8: every quantized layer, chained.

    Layer i reads layer i-1's output buffer whenever its element count allows
    (``workloads.chain_sources``; the glue between U-Net layers is not part of
    the pass), else a seeded N(0, 1) buffer of its own.  Codebooks have the
    unit-scale standard deviation, so activations stay near unit scale along
    the chain.  One step = one whole pass, replayed from a HIP graph.
    """
    import numpy as np

    layers = W.sweep_layers(full=a.full)
    M = {"W2": 2, "W4": 4, "W2K": 2, "W4K": 4}[a.variant]
    kaq = a.variant.endswith("K")       # 3x3 convolutions in the kernel-aware format (g = 9)
    src = W.chain_sources(layers, batch=8)
    branch = W.branch_inputs(layers)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(W.SEED_BASE + 4)
    specs, seeds, objs, items = [], [], [], []
    total_flops = total_bytes = 0
    prev_y = None
    for i, lay in enumerate(layers):
        spec = W.sweep_spec(lay, M, batch=8, g=9 if kaq and lay.kind == "conv3x3" else 8, codebook_std="chain")
        seed = W.SEED_BASE + 100 + i
        wts = W.generate(spec.with_n(1), seed)         # weights are drawn before activations
        layer = P.AQLayer(spec, wts, max_tokens=spec.tokens)
        xshape = layer.in_shape(spec.n)
        if branch[i] is not None:
            x = objs[branch[i]][1]                     # the block input, which its first conv reads too
            assert tuple(x.shape) == tuple(xshape), (spec.name, x.shape, xshape)
        elif src[i] is not None:
            x = prev_y.view(xshape)
        else:
            x = torch.randn(xshape, generator=gen, device="cuda", dtype=torch.float32).to(torch.float16)
        y = torch.empty(layer.out_shape(spec.n), dtype=torch.float16, device="cuda")
        fn = (lambda layer=layer, x=x, y=y: layer.forward(x, None, out=y))
        specs.append(spec)
        seeds.append(seed)
        objs.append((layer, x, y))
        items.append((layer, fn))
        total_flops += spec.dense_flops
        total_bytes += algorithmic_bytes(spec)
        prev_y = y

    def run_pass():
        for _, fn in items:
            fn()

    layer_objs, layer_ns = [it[0] for it in items], [sp.n for sp in specs]

    def decode_all():
        P.AQLayer.prepare_all(layer_objs, layer_ns)

    def run_pass_batched():
        # every record decode of the pass first, one launch per records kernel
        # and 32 layers (aq_layers_prepare), then the forwards, each of which
        # launches its product only; the decodes stay inside the timed pass
        decode_all()
        run_pass()

    side_b = torch.cuda.Stream()
    fns = [fn for _, fn in items]

    def run_pass_two_streams():
        # the batched decodes, then the pass with every residual skip
        # convolution on a second stream beside its block's 3x3 convolutions
        run_pass_branches(torch, fns, branch, side_b, first=decode_all)

    side = torch.cuda.Stream()

    def run_pass_overlapped():
        # every forward's weight records (where its route has them) decoded on a
        # second stream, in layer order, overlapped with the products of earlier
        # layers; each forward waits for its own layer's records only
        main = torch.cuda.current_stream()
        ahead = a.records_ahead

        def prep(j):
            side.wait_stream(main)              # issued once layer j - ahead's forward is queued
            items[j][0].prepare(specs[j].n, stream=side.cuda_stream)
            ev = torch.cuda.Event()
            ev.record(side)
            return ev

        ready = {j: prep(j) for j in range(min(ahead, len(items)))}
        for i, (_, fn) in enumerate(items):
            main.wait_event(ready.pop(i))
            if i + ahead < len(items):
                ready[i + ahead] = prep(i + ahead)
            fn()
        main.wait_stream(side)

    def time_graph(body, extra_trials=0):
        stream = torch.cuda.Stream()
        stream.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(stream):
            body()
        torch.cuda.current_stream().wait_stream(stream)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.stream(stream):
            with torch.cuda.graph(g, stream=stream):
                body()
        torch.cuda.current_stream().wait_stream(stream)
        for _ in range(max(0, a.warmup)):
            g.replay()
        torch.cuda.synchronize()
        times = []
        for _ in range(1 + extra_trials):
            # the first trial is the timed steps; extra trials repeat them for the spread
            t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            t0.record()
            for _ in range(a.steps):
                g.replay()
            t1.record()
            torch.cuda.synchronize()
            times.append(t0.elapsed_time(t1) * 1e3 / a.steps)
        return (times[0], times) if extra_trials else times[0]

    # the timed steps: whole passes replayed from one graph on one stream;
    # --records-overlap also times the schedule that decodes records on a
    # second stream ahead of their forwards (measured slower: the replayed
    # graph's cross-stream dependencies cost more than they hide)
    batched = a.records == "batched"
    serial_us, serial_trials = time_graph(run_pass_batched if batched else run_pass, extra_trials=4)
    other_us = time_graph(run_pass if batched else run_pass_batched)
    two_us = time_graph(run_pass_two_streams) if batched else None
    pass_us = two_us if (batched and a.streams == 2) else serial_us
    trials_us = serial_trials if pass_us == serial_us else [pass_us]
    overlap_us = time_graph(run_pass_overlapped) if a.records_overlap else None
    decode_us = time_graph(decode_all)          # the batched decodes alone
    run_pass()                                  # consumes the preparations the last capture left pending
    torch.cuda.synchronize()

    # per-launch kernel durations inside the same pass (events around every launch)
    per_layer, tmode, pass_us_ev = launch_times(torch, items)

    # the same products as dense fp16 GEMMs in the vendor library (comparator)
    dense_ref = None
    if not a.no_dense_ref:
        dfns = dense_gemm_reference(torch, specs, gen)
        dense_pass_us = time_graph(lambda: [f() for f in dfns])
        dense_layer_us = [_graph_time_us(torch, f, reps=10) for f in dfns]
        dense_ref = {"kind": "torch.matmul fp16 (hipBLASLt): every layer's [tokens x K] x [K x C_out] product, "
                             "seeded N(0, 1) operands, weights stored [C_out, K], im2col not counted",
                     "ms_per_step": round(dense_pass_us / 1e3, 6),
                     "value": round(total_flops / (dense_pass_us * 1e-6) / 1e12, 3),
                     "aq_pass_speedup": round(dense_pass_us / pass_us, 3)}

    # weight source of every forward: in-loop decode (W never in memory), records
    # (the decompress-then-compute route: unscaled fp16 W written and read back
    # every forward) or the table path; then the same pass with the in-loop
    # decode forced wherever the format has one
    src_t, src_n, rec_bytes = {}, {}, 0
    for i, (layer, _) in enumerate(items):
        d = layer.describe(specs[i].n)
        k = "table" if d.get("path") == "lut" else "records" if d.get("weights") == "records" else "in-loop"
        src_t[k] = src_t.get(k, 0.0) + sum(t for _, t in per_layer[i])
        src_n[k] = src_n.get(k, 0) + 1
        rec_bytes += int(d.get("records_bytes", 0))
    for layer, _ in items:
        layer.set_option("weights", 1)
    n_inloop = sum(1 for i, (layer, _) in enumerate(items) if layer.describe(specs[i].n).get("weights") != "records")
    inloop_us = time_graph(run_pass)
    for layer, _ in items:
        layer.set_option("weights", 0)
    ttot = sum(src_t.values())
    weights = {"time_frac": {k: round(v / ttot, 4) for k, v in sorted(src_t.items())},
               "layers": dict(sorted(src_n.items())), "record_bytes_per_pass": rec_bytes,
               "in_loop_pass": {"ms_per_step": round(inloop_us / 1e3, 6),
                                "value": round(total_flops / (inloop_us * 1e-6) / 1e12, 3),
                                "layers_in_loop": n_inloop,
                                "note": "the same pass with the in-loop decode forced on every layer whose format "
                                        "has one: W is never written to memory"}}
    flops = [sp.dense_flops for sp in specs]
    kname, k_us, k_n, k_flops, ktable = dominant_kernel(per_layer, flops)
    workload = f"unet_sweep_b8_{a.variant}{'_full' if a.full else ''}_chained"
    k_tflops = k_flops / (k_us * 1e-6) / 1e12
    # every layer's output at unit scale (no overflow, no collapse along the chain)
    rms = [float(y.float().pow(2).mean().sqrt()) for _, _, y in objs]

    if a.table:
        with open(a.table, "w") as f:
            fmt = "g=9 for 3x3 convolutions, g=8 elsewhere" if kaq else "g=8"
            f.write(f"# U-Net pass, batch 8, {a.variant} ({fmt}, M={M}, B=8), fp16, chained\n\n")
            f.write(f"Command: `python bench.py --config sweep --variant {a.variant}"
                    f"{' --full' if a.full else ''} --table <this file>`\n\n")
            f.write(f"{len(layers)} layers, {sum(s is not None and b is None for s, b in zip(src, branch))} reading the "
                    f"previous layer's output, {sum(b is not None for b in branch)} (residual skips) their block's "
                    f"input; "
                    f"{total_flops / 1e9:.1f} dense-equivalent GFLOP.  Whole pass in one HIP graph: "
                    f"{pass_us:.1f} us ({total_flops / (pass_us * 1e-6) / 1e12:.1f} TFLOP/s, "
                    f"{total_flops / (pass_us * 1e-6) / 1e12 / PEAK_MFMA_F16_TFLOPS:.3f} of 2.5 PFLOP/s; "
                    f"record decodes {'batched at the start of the pass' if batched else 'in each forward'}"
                    f"{', residual skip convolutions on a second stream' if pass_us == two_us else ''}; "
                    + (f"all on one stream: {serial_us:.1f} us; " if pass_us == two_us else
                       f"residual skips on a second stream: {two_us:.1f} us; " if two_us is not None else "")
                    + f"with the decodes {'in each forward' if batched else 'batched'}: {other_us:.1f} us; the batched "
                    f"decodes alone: {decode_us:.1f} us).  "
                    f"Per-layer times below: each forward alone in a HIP graph (sum "
                    f"{sum(t for lay in per_layer for _, t in lay):.1f} us), split among its launches by "
                    f"timing events (eager pass with events: {pass_us_ev:.1f} us)." +
                    ("" if overlap_us is None else
                     f"  With record decodes on a second stream {a.records_ahead} layer(s) ahead: {overlap_us:.1f} us.")
                    + "\n\n")
            f.write("Weight source (share of the per-layer time; layers): " +
                    ", ".join(f"{k} {weights['time_frac'][k]:.3f} ({weights['layers'][k]})" for k in weights["layers"]) +
                    f"; records written and read back per pass: {rec_bytes / 1e6:.1f} MB.  The same pass with the "
                    f"in-loop decode forced wherever the format has one ({n_inloop} of {len(items)} layers; W never in "
                    f"memory): {inloop_us:.1f} us ({total_flops / (inloop_us * 1e-6) / 1e12:.1f} TFLOP/s).\n\n")
            if dense_ref is not None:
                f.write(f"Dense fp16 comparator ({dense_ref['kind']}): the pass's products in one graph "
                        f"{dense_pass_us:.1f} us ({dense_ref['value']:.1f} TFLOP/s); the AQ pass is "
                        f"{dense_ref['aq_pass_speedup']:.2f}x that speed.\n\n")
            f.write("Per kernel (sum over the pass):\n\n| kernel | launches | total us | share | TFLOP/s |\n"
                    "|---|---|---|---|---|\n")
            ksum = sum(r[1] for r in ktable)
            for n, t, c, fl in ktable:
                f.write(f"| `{n}` | {c} | {t:.1f} | {t / ksum:.3f} | "
                        f"{(fl / (t * 1e-6) / 1e12) if fl else 0:.1f} |\n")
            f.write("\nPer layer (kernels in launch order, us each):\n\n"
                    "| layer | kind | tokens | K | C_out | input | launches | us | TFLOP/s | out rms | dense fp16 GEMM us |\n"
                    "|---|---|---|---|---|---|---|---|---|---|---|\n")
            for i, (lay, sp) in enumerate(zip(layers, specs)):
                us = sum(t for _, t in per_layer[i])
                ks = " + ".join(f"`{n.split('<')[0]}` {t:.1f}" for n, t in per_layer[i])
                f.write(f"| {sp.name} | {lay.kind}{' s2' if lay.stride == 2 else ''} | {sp.tokens} | {sp.K} | "
                        f"{sp.C_out} | {'block input' if branch[i] is not None else 'prev' if src[i] is not None else 'own'}"
                        f" | {ks} | {us:.2f} | "
                        f"{sp.dense_flops / (us * 1e-6) / 1e12:.1f} | {rms[i]:.3f} | "
                        f"{'' if dense_ref is None else f'{dense_layer_us[i]:.2f}'} |\n")
    out = {
        "metric": "dense-equivalent TFLOP/s of the AQ layer forward",
        "value": round(total_flops / (pass_us * 1e-6) / 1e12, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(pass_us / 1e3, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic (seeded; LDM-4-shaped U-Net layers at batch 8, random codebooks/codes/activations, "
                "chained where shapes allow)",
        "config": {"workload": workload, "layers": len(layers),
                   "chained_inputs": sum(s is not None and b is None for s, b in zip(src, branch)),
                   "branch_inputs": sum(b is not None for b in branch),
                   "launch": "hip graph of the whole pass", "format": f"{a.variant}: g={9 if kaq else 8}/8, M={M}, B=8"},
        "hbm_gbs_algorithmic": round(total_bytes / (pass_us * 1e-6) / 1e9, 3),
        "algorithmic_bytes": total_bytes,
        "dense_flops": total_flops,
        "roofline": {"bound": "mfma", "achieved": round(k_tflops, 3), "peak": PEAK_MFMA_F16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(k_tflops / PEAK_MFMA_F16_TFLOPS, 4),
                     "traffic": measured_traffic_kernel(workload, kname), "kernel": kname, "launches": k_n,
                     "kernel_avg_us": round(k_us / k_n, 3), "kernel_flops": k_flops, "timing": tmode,
                     "pass_frac": round(total_flops / (pass_us * 1e-6) / 1e12 / PEAK_MFMA_F16_TFLOPS, 4)},
        "kernels": [{"kernel": n, "launches": c, "total_us": round(t, 2)} for n, t, c, _ in ktable[:6]],
        "weights": weights,
        "schedule": {"streams": 2 if pass_us == two_us else 1, "records": a.records,
                     "ms_per_step_two_streams": None if two_us is None else round(two_us / 1e3, 6),
                     "ms_per_step_records_batched": round((serial_us if batched else other_us) / 1e3, 6),
                     "ms_per_step_records_per_forward": round((other_us if batched else serial_us) / 1e3, 6),
                     "batched_decodes_us": round(decode_us, 2),
                     "ms_per_step_records_ahead": None if overlap_us is None else round(overlap_us / 1e3, 6),
                     "records_ahead": a.records_ahead if a.records_overlap else None,
                     "note": "records batched: every record decode of the pass launched first, one launch per "
                             "records kernel and 32 layers (aq_layers_prepare), then the forwards; per_forward: each "
                             "forward decodes its own; records_ahead: per-forward decodes on a second stream, that "
                             "many layers ahead (aq_layer_prepare); every decode is inside the timed pass"},
        "activation_rms": [round(min(rms), 4), round(max(rms), 4)],
        "trials": {"n": len(trials_us), "median_ms": round(statistics.median(trials_us) / 1e3, 6),
                   "min_ms": round(min(trials_us) / 1e3, 6),
                   "note": "the timed steps, then the same steps repeated, each trial a.steps graph replays"},
        "dense_reference": dense_ref,
    }
    if a.copy_bytes > 0:
        src_b = torch.empty(a.copy_bytes, dtype=torch.uint8, device="cuda")
        torch.empty_like(src_b).copy_(src_b)
        torch.cuda.synchronize()
    if not a.no_cpu_baseline:
        out["cpu_baseline"] = sweep_cpu_baseline(specs, seeds)
    for layer, _, _ in objs:
        layer.close()
    return out


def lut_regime_bench(a, torch, P, W):
    """Table path vs matrix-core path for few tokens on U-Net linear shapes (fp16, B = 8).

    Each (K, C_out, M) layer is timed at every token count with both paths
    forced.  Warm: the same layer back to back in a HIP graph (weights stay in
    L2 / MALL).  Rotated (the layers whose codes are at least 2 MB): a graph
    of forwards over R copies of the layer at distinct device addresses, R
    copies holding at least 640 MB of codes (over twice the 256 MB MALL), so
    every forward reads its codes from HBM.  Algorithmic bytes: codes +
    codebooks + scales + X + Y.  The launch floor is a one-element kernel
    replayed in the same kind of graph.
    """
    import numpy as np

    ns = tuple(int(v) for v in a.lut_ns.split(",")) if a.lut_ns else (1, 2, 4, 8, 16, 32)
    shapes = sorted(set((s.K, s.C_out, s.M) for s in W.lut_regime_specs()))
    if a.lut_k:
        shapes = [sh for sh in shapes if sh[0] == a.lut_k]
    if a.lut_m:
        shapes = [sh for sh in shapes if sh[2] == a.lut_m]
    tiny = torch.zeros(1, device="cuda")
    floor_us = _graph_time_us(torch, lambda: tiny.add_(1.0), reps=20)
    rows = []
    for K, C, M in shapes:
        base = W.LayerSpec(name=f"lut_{K}to{C}_M{M}", C_out=C, K=K, g=8, M=M, B=8, n=max(ns))
        inp = W.generate(base, W.SEED_BASE + 200 + len(rows))
        code_bytes = C * (K // 8) * M
        R = int(np.ceil(640e6 / code_bytes)) if code_bytes >= 2e6 else 0
        layers = [P.AQLayer(base, inp, max_tokens=max(ns)) for _ in range(max(1, R))]
        xfull = torch.from_numpy(inp["x"]).cuda()
        for n in ns:
            spec = base.with_n(n)
            x = xfull[:n].contiguous()
            y = torch.empty((n, C), dtype=torch.float16, device="cuda")
            t, tr = {}, {}
            for path in ("lut", "decode"):
                for L in layers:
                    L.set_path(path)
                t[path] = _graph_time_us(torch, lambda: layers[0].forward(x, None, out=y), reps=20)
                if R:
                    tr[path] = _graph_time_us(torch, lambda: [L.forward(x, None, out=y) for L in layers], reps=1,
                                              trials=3) / R
            for L in layers:
                L.set_path("auto")
            rows.append((K, C, M, n, t["lut"], t["decode"], tr.get("lut"), tr.get("decode"), algorithmic_bytes(spec),
                         layers[0].choose_path(n)))
        for L in layers:
            L.close()
    if a.table:
        with open(a.table, "w") as f:
            f.write("# Table (LUT) path vs matrix-core path at few tokens, fp16, g=8, B=8\n\n")
            f.write("Command: `python bench.py --config lutregime --table <this file>`\n\n")
            f.write("GB/s are algorithmic bytes (codes, codebooks, scales, X, Y) over the table-path time.  Warm: the "
                    "same layer replayed in a HIP graph (its codes stay in L2 / MALL).  Rotated: one graph over "
                    "copies of the layer holding >= 640 MB of codes, so each forward reads its codes from HBM "
                    "(layers with >= 2 MB of codes).  Launch floor (a one-element kernel, same graph replay): "
                    f"{floor_us:.2f} us per launch.\n\n")
            f.write("| K | C_out | M | tokens | table us | table GB/s | table us rotated | table GB/s rotated | "
                    "matrix-core us | matrix-core us rotated | faster | dispatch |\n"
                    "|---|---|---|---|---|---|---|---|---|---|---|---|\n")
            for K, C, M, n, tl, td, tlr, tdr, ab, ch in rows:
                faster = "table" if (tlr or tl) < (tdr or td) else "matrix-core"
                f.write(f"| {K} | {C} | {M} | {n} | {tl:.2f} | {ab / tl / 1e3:.0f} | "
                        f"{'' if tlr is None else f'{tlr:.2f}'} | {'' if tlr is None else f'{ab / tlr / 1e3:.0f}'} | "
                        f"{td:.2f} | {'' if tdr is None else f'{tdr:.2f}'} | {faster} | {ch} |\n")
    rot = [r for r in rows if r[6] is not None]
    best = max(rot, key=lambda r: r[8] / r[6]) if rot else max(rows, key=lambda r: r[8] / r[4])
    t_best = best[6] if rot else best[4]
    gbs = best[8] / t_best / 1e3
    return {
        "metric": "dense-equivalent TFLOP/s and HBM GB/s of AQ layer forward (table path)",
        "value": round(gbs, 3),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": 3,
        "warmup": 1,
        "ms_per_step": round(t_best / 1e3, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded; U-Net linear shapes at few tokens)",
        "config": {"workload": f"lut_{best[0]}to{best[1]}_M{best[2]}_n{best[3]}", "path": "lut",
                   "launch": "hip graph over rotated weight copies" if rot else "hip graph of 20 steps",
                   "cases": len(rows), "launch_floor_us": round(floor_us, 3)},
        "roofline": {"bound": "hbm", "achieved": round(gbs, 3), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(gbs / PEAK_HBM_GBS, 4), "traffic": None, "kernel": "lut_fwd_kernel"},
    }


def grad_bench(a, torch, P, W):
    """One step = one codebook gradient (weight gradient on the matrix cores plus the code-indexed gather).

    The workload is the named layer with fp16 X and dY (an int8 forward input is
    replaced by fp16 values of the same shape).  FLOPs are those of dY^T X,
    2 per multiply-accumulate, the same count as the forward.
    """
    import dataclasses

    import numpy as np

    spec = W.config_spec(a.config)
    if spec.x_dtype != "f16":
        spec = dataclasses.replace(spec, x_dtype="f16")
    inp = W.generate(spec, W.SEED_BASE + 100)
    gi = W.generate_grad_inputs(spec, W.SEED_BASE + 101, "f16")
    layer = P.AQLayer(spec, inp)
    x = torch.from_numpy(np.ascontiguousarray(gi["x"])).cuda()
    dy = torch.from_numpy(np.ascontiguousarray(gi["dy"])).cuda()
    dC = torch.empty((spec.M, 1 << spec.B, spec.g), dtype=torch.float32, device="cuda")
    for _ in range(max(1, a.warmup)):
        layer.codebook_grad(x, dy, out=dC)       # the first call prepares the code index
    torch.cuda.synchronize()
    per_graph = max(1, min(a.steps, 50))
    reps = (a.steps + per_graph - 1) // per_graph
    us = _graph_time_us(torch, lambda: layer.codebook_grad(x, dy, out=dC), per_graph, trials=reps)
    ms = us * 1e-3
    if a.copy_bytes > 0:
        src = torch.empty(a.copy_bytes, dtype=torch.uint8, device="cuda")
        torch.empty_like(src).copy_(src)
        torch.cuda.synchronize()
    flops = spec.dense_flops
    tflops = flops / (ms * 1e-3) / 1e12
    out = {
        "metric": "dense-equivalent TFLOP/s of the AQ codebook gradient",
        "value": round(tflops, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": reps * per_graph,
        "warmup": a.warmup,
        "ms_per_step": round(ms, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic (seeded; LDM-4-shaped layer, random codes, fp16 activations and output gradients)",
        "config": {"workload": spec.name + "_codebook_grad", "launch": f"hip graph of {per_graph} steps",
                   "tokens": spec.tokens, "K": spec.K, "C_out": spec.C_out, "g": spec.g, "M": spec.M, "B": spec.B},
        "dense_flops": flops,
        # both launches of a step (weight gradient, then gather); the kernel
        # trace splits them
        "roofline": {"bound": "mfma", "achieved": round(tflops, 3), "peak": PEAK_MFMA_F16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(tflops / PEAK_MFMA_F16_TFLOPS, 4), "traffic": None, "kernel_us": round(us, 3)},
    }
    if not a.no_cpu_baseline:
        import oracle as O
        ginp = {"codes": inp["codes"], "scales": inp["scales"], "x": gi["x"]}
        t0 = time.perf_counter()
        O.codebook_grad(spec, ginp, gi["dy"], x_dtype="f16", dy_dtype="f16")
        t = time.perf_counter() - t0
        try:
            from threadpoolctl import threadpool_info
            threads = max((p.get("num_threads", 1) for p in threadpool_info()), default=1)
        except Exception:
            threads = os.cpu_count() or 1
        out["cpu_baseline"] = {"value": round(flops / t / 1e12, 6), "unit": "TFLOP/s", "cores": int(threads),
                               "kind": "oracle",
                               "sample": f"whole layer ({spec.name}): fp64 dY^T X (BLAS) + scatter-add, one run, "
                                         f"{t:.3f} s"}
    layer.close()
    return out


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed steps (default 20 passes, 200 forwards)")
    ap.add_argument("--warmup", type=int, default=None, help="untimed steps (default 3 passes, 20 forwards)")
    ap.add_argument("--config", default="sweep", help="sweep (default), lutregime, or one layer: tiny, conv64, "
                                                      "qkv16, conv8")
    ap.add_argument("--path", default="auto", choices=["auto", "lut", "decode"])
    ap.add_argument("--weights", default="auto", choices=["auto", "in-loop", "records"],
                    help="one layer: the decode path's weight source (in-loop: W never in memory; records: the "
                         "unscaled decoded weights written and read back every forward)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-dense-ref", action="store_true",
                    help="sweep: skip the dense fp16 GEMM comparator (torch.matmul on the same shapes)")
    ap.add_argument("--no-graph", action="store_true", help="launch every step from Python instead of a HIP graph")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="after timing, run one plain device copy of this many bytes (counter calibration)")
    ap.add_argument("--variant", default="W2", choices=["W2", "W4", "W2K", "W4K"],
                    help="sweep: M = 2 or 4 codebooks of 256 (K: 3x3 convolutions with g = 9, one group per filter)")
    ap.add_argument("--full", action="store_true", help="sweep: every linear of the transformer blocks")
    ap.add_argument("--table", default="", help="sweep: write the per-layer table (markdown) here")
    ap.add_argument("--lut-ns", default="", help="lutregime: token counts, comma separated (default 1..32)")
    ap.add_argument("--lut-k", type=int, default=0, help="lutregime: only the shapes with this K")
    ap.add_argument("--lut-m", type=int, default=0, help="lutregime: only the shapes with this M")
    ap.add_argument("--records-ahead", type=int, default=1,
                    help="sweep: layers ahead of the current forward whose records the second stream decodes")
    ap.add_argument("--records", default="batched", choices=["batched", "per-forward"],
                    help="sweep: the timed pass decodes every layer's records first in batched launches "
                         "(aq_layers_prepare), or each forward decodes its own")
    ap.add_argument("--streams", type=int, default=1, choices=[1, 2],
                    help="sweep: the timed pass in layer order on one stream (1), or with every residual skip "
                         "convolution on a second stream beside its block's 3x3 convolutions (2, with --records "
                         "batched; measured slower: the graph's cross-stream edges cost more than the overlap "
                         "hides); both are always timed and reported")
    ap.add_argument("--records-overlap", action="store_true",
                    help="sweep: also time the pass with record decodes on a second stream (--records-ahead)")
    ap.add_argument("--op", default="forward", choices=["forward", "grad"],
                    help="grad: the codebook gradient of the named layer instead of its forward")
    a = ap.parse_args(argv)

    if a.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {a.gpus}): the AQ layer forward here runs each "
              "layer on one GPU and is not sharded across GPUs", file=sys.stderr)
        return 2

    if a.steps is None:
        a.steps = 20 if a.config == "sweep" else 200
    if a.warmup is None:
        a.warmup = 3 if a.config == "sweep" else 20
    if a.steps < 1:
        print("--steps must be >= 1", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import paper_2506_05960_amd as P
    import workloads as W

    P.load_library()
    torch.cuda.set_device(0)
    if a.config == "sweep":
        print(json.dumps(sweep_bench(a, torch, P, W)), flush=True)
        return 0
    if a.config == "lutregime":
        print(json.dumps(lut_regime_bench(a, torch, P, W)), flush=True)
        return 0
    if a.op == "grad":
        print(json.dumps(grad_bench(a, torch, P, W)), flush=True)
        return 0
    spec = W.config_spec(a.config)
    inp = W.config_inputs(a.config)
    layer = P.AQLayer(spec, inp)
    if a.path != "auto":
        layer.set_path(a.path)
    if a.weights != "auto":       # the decode path's weight source forced (AQ_OPT_WEIGHTS)
        layer.set_option("weights", 1 if a.weights == "in-loop" else 2)
    wsuffix = "" if a.weights == "auto" else "_" + a.weights.replace("-", "")
    path = layer.choose_path(spec.tokens)
    x = torch.from_numpy(np.ascontiguousarray(inp["x"])).cuda()
    xs = None if inp["x_scales"] is None else torch.from_numpy(inp["x_scales"]).cuda()
    y = torch.empty(layer.out_shape(spec.n), dtype=torch.float16 if spec.y_dtype == "f16" else torch.float32,
                    device="cuda")

    for _ in range(a.warmup):
        layer.forward(x, xs, out=y)
    torch.cuda.synchronize()

    # The forward allocates nothing and issues no memset, so runs of steps can
    # be captured in HIP graphs and replayed: the timed region then measures
    # the GPU, not Python's per-launch overhead.  Exactly a.steps steps are
    # timed: a graph of up to 50 forwards replayed a.steps // 50 times, then
    # one graph of the remaining a.steps % 50.
    per_graph = max(1, min(a.steps, 50))
    nfull, tail = divmod(a.steps, per_graph)

    def capture(n):
        stream = torch.cuda.Stream()
        stream.wait_stream(torch.cuda.current_stream())
        g = torch.cuda.CUDAGraph()
        with torch.cuda.stream(stream):
            with torch.cuda.graph(g, stream=stream):
                for _ in range(n):
                    layer.forward(x, xs, out=y)
        torch.cuda.current_stream().wait_stream(stream)
        g.replay()
        torch.cuda.synchronize()
        return g

    graph = tail_graph = None
    if not a.no_graph:
        graph = capture(per_graph)
        if tail:
            tail_graph = capture(tail)
    steps = a.steps

    def timed_steps():
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record()
        if graph is not None:
            for _ in range(nfull):
                graph.replay()
            if tail_graph is not None:
                tail_graph.replay()
        else:
            for _ in range(steps):
                layer.forward(x, xs, out=y)
        stop.record()
        torch.cuda.synchronize()
        return start.elapsed_time(stop) / steps

    ms = timed_steps()
    trials_ms = [ms] + [timed_steps() for _ in range(4)]     # the timed steps, then four repeats for the spread

    # The dominant kernel's own duration: timing events around every launch of
    # ten forwards in one graph (a pre-decoded forward is two launches, records
    # then product; a table-path forward is table+gather then reduction).
    per_layer, tmode, _ = launch_times(torch, [(layer, lambda: layer.forward(x, xs, out=y))] * 10)
    flops = spec.dense_flops
    kname, k_us_tot, k_n, k_flops, ktable = dominant_kernel(per_layer, [flops] * len(per_layer))
    kms = k_us_tot / k_n / 1e3
    tflops = flops / (ms * 1e-3) / 1e12
    gbs = algorithmic_bytes(spec) / (ms * 1e-3) / 1e9
    k_tflops = (k_flops / k_n) / (kms * 1e-3) / 1e12
    k_gbs = algorithmic_bytes(spec) / (kms * 1e-3) / 1e9
    if a.copy_bytes > 0:
        src = torch.empty(a.copy_bytes, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
    traffic = measured_traffic_kernel(a.config + wsuffix, kname)
    if path == "decode" and spec.tile_dtype != "f32":
        roof = {"bound": "mfma", "achieved": round(k_tflops, 3), "peak": PEAK_MFMA_F16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(k_tflops / PEAK_MFMA_F16_TFLOPS, 4), "traffic": traffic}
    elif path == "decode":
        roof = {"bound": "alu", "achieved": round(k_tflops, 3), "peak": PEAK_F32_VALU_TFLOPS, "unit": "TFLOP/s",
                "frac": round(k_tflops / PEAK_F32_VALU_TFLOPS, 4), "traffic": traffic}
    else:
        roof = {"bound": "hbm", "achieved": round(k_gbs, 3), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(k_gbs / PEAK_HBM_GBS, 4), "traffic": traffic}
    roof["kernel"] = kname
    roof["kernel_avg_us"] = round(kms * 1e3, 3)
    roof["timing"] = tmode

    out = {
        "metric": "dense-equivalent TFLOP/s of the AQ layer forward",
        "value": round(tflops, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": a.warmup,
        "ms_per_step": round(ms, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": spec.tile_dtype if path == "decode" else "f32",
        "data": "synthetic (seeded; LDM-4-shaped layer, random codebooks/codes/activations)",
        "config": {"workload": spec.name + wsuffix, "path": path, "launch": "eager" if graph is None else f"hip graph of {per_graph} steps", "tokens": spec.tokens, "K": spec.K, "C_out": spec.C_out,
                   "g": spec.g, "M": spec.M, "B": spec.B, "x_dtype": spec.x_dtype, "y_dtype": spec.y_dtype},
        "hbm_gbs_algorithmic": round(gbs, 3),
        "algorithmic_bytes": algorithmic_bytes(spec),
        "dense_flops": flops,
        "roofline": roof,
        "trials": {"n": len(trials_ms), "median_ms": round(statistics.median(trials_ms), 6),
                   "min_ms": round(min(trials_ms), 6),
                   "note": "the timed steps, then the same steps repeated four times"},
        "kernels": [{"kernel": n, "launches": c // 10, "avg_us": round(t / c, 3)} for n, t, c, _ in ktable],
    }
    if path == "decode":
        # weight source of this forward; on the records route (W written to
        # memory every forward) the in-loop decode (W never in memory) is timed
        # beside it the same way
        d = layer.describe(spec.n)
        wsrc = {"source": "records" if d.get("weights") == "records" else "in-loop",
                "record_bytes": int(d.get("records_bytes", 0))}
        if wsrc["source"] == "records":
            layer.set_option("weights", 1)
            if layer.describe(spec.n).get("weights") != "records":
                g_il = capture(per_graph)
                t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                t0.record()
                for _ in range(max(1, nfull)):
                    g_il.replay()
                t1.record()
                torch.cuda.synchronize()
                ms_il = t0.elapsed_time(t1) / (max(1, nfull) * per_graph)
                wsrc["in_loop"] = {"ms_per_step": round(ms_il, 6), "value": round(flops / (ms_il * 1e-3) / 1e12, 3),
                                   "route": layer.describe(spec.n).get("route"),
                                   "tile": layer.describe(spec.n).get("tile")}
            layer.set_option("weights", 0)
        out["weights"] = wsrc
    if not a.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(spec, inp)
    layer.close()
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
