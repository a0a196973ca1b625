"""Benchmark: the Qwen3-8B decode-step linear stack as packed ternary GEMVs.

One step = every packed linear of one decode step at batch 1: 36 layers x
{q, k, v, o, gate, up, down} (252 matrices, 6.95 G weights) as 144 dependent
stages (q+k+v grouped, o, gate+up grouped, down), run as one tq_gemv_chain
launch per step; the same step as 144 launches in a HIP graph is reported
beside it (outputs compared bit for bit).  Inputs are seeded
synthetic stand-ins for the paper's converted weights (shapes of section 3,
10% two-plane groups) and stay resident in HBM; the 1.70 GB of packed weights
is far larger than the caches, so every step streams them from HBM.

Prints one JSON line: value = aggregate GB/s of algorithmic bytes (packed
weights + activations + outputs) per step time, plus ms_per_step, the
roofline of chain_kernel (one launch per step: its duration is the HIP-event
timed region on the launch stream over the launches it holds), the measured
streaming-read ceiling at the same byte count and the CPU oracle timed on a
bounded sample (all host cores and one thread).

    python bench.py [--gpus 1] [--steps 20] [--warmup 3] [--layers 36]
    python bench.py --extra     # also: small batch, codec, and the 4096 x 2560
                                # comparison with dense fp16 (one JSON line each)
"""

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
COPY_BYTES = 256 << 20      # calibration copy: 256 MiB read + 256 MiB written


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def build_stack(layers, device, paper_representation=False):
    """Generate (host threads) and pack (GPU) every projection of the stack.
    With ``paper_representation``: an offset on every group and the paper's
    3.6% two-plane groups instead of the benchmark's 10%."""
    from concurrent.futures import ThreadPoolExecutor

    import torch

    from paper_2609_09240_amd import synth, tq
    names = [n for n, _, _ in synth.PROJECTIONS]
    mats, xs = [], []
    t0 = time.time()
    if paper_representation:
        gen = lambda layer: [synth.projection(n, layer, cfg=3, f2=synth.PAPER_TWO_PLANE, offset0=True)  # noqa: E731
                             for n in names]
    else:
        gen = lambda layer: [synth.projection(n, layer, cfg=3) for n in names]  # noqa: E731
    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        pending = [ex.submit(gen, layer) for layer in range(min(layers, 8))]
        for layer in range(layers):
            inputs = pending[layer].result()
            pending[layer] = None
            if layer + 8 < layers:
                pending.append(ex.submit(gen, layer + 8))
            mats.append({n: tq.PackedLinear.from_inputs(inp, device) for n, inp in zip(names, inputs)})
            xs.append([torch.from_numpy(synth.stage_activations(s, layer, cfg=3)).to(device)
                       for s in range(len(synth.STAGES))])
            if layer % 6 == 5 or layer == layers - 1:
                torch.cuda.synchronize()
                log(f"built layers 0..{layer} ({time.time() - t0:.1f} s)")
    return mats, xs


def step_launches(mats, xs):
    """The launches of one decode step, in dependency order."""
    from paper_2609_09240_amd import synth
    out = []
    for layer in range(len(mats)):
        for s, names in enumerate(synth.STAGES):
            out.append(([mats[layer][n] for n in names], xs[layer][s]))
    return out


def time_stack(mats, xs, steps, warmup):
    """Capture one decode step of the stack in a HIP graph, replay it
    `warmup` times, then time `steps` replays; returns (ms per step,
    launches, graph, outputs)."""
    import torch

    from paper_2609_09240_amd import tq
    launches = step_launches(mats, xs)
    dev = xs[0][0].device
    outs = [[torch.empty(m.n_out, dtype=torch.float16, device=dev) for m in ms] for ms, _ in launches]
    stream = torch.cuda.Stream()

    def run_step():
        for (ms, x), ys in zip(launches, outs):
            if len(ms) == 1:
                tq.tq_gemv(ms[0], x, y=ys[0], stream=stream)
            else:
                tq.tq_gemv_grouped(ms, x, ys=ys, stream=stream)

    with torch.cuda.stream(stream):
        run_step()                                  # first launches outside capture
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        run_step()
    torch.cuda.synchronize()
    for _ in range(warmup):
        graph.replay()
    torch.cuda.synchronize()
    t_start = torch.cuda.Event(enable_timing=True)
    t_stop = torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(stream):
        t_start.record(stream)
        for _ in range(steps):
            graph.replay()
        t_stop.record(stream)
    torch.cuda.synchronize()
    ms_per_step = t_start.elapsed_time(t_stop) / steps
    # Spread: the same number of replays again, each between its own pair
    # of events (outside the timed region above).
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    with torch.cuda.stream(stream):
        for a, b in evs:
            a.record(stream)
            graph.replay()
            b.record(stream)
    torch.cuda.synchronize()
    per_step = sorted(a.elapsed_time(b) * 1e3 for a, b in evs)
    time_stack.spread_us = {q: round(per_step[min(len(per_step) - 1, int(q / 100 * len(per_step)))], 2)
                            for q in (10, 50, 90)}
    return ms_per_step, launches, graph, outs


def time_chain(mats, xs, steps, warmup):
    """The same decode step as one tq_gemv_chain launch per step (every
    stage waits for the previous one inside the launch); HIP events on the
    launch stream around `steps` calls.  Returns (ms per step, chain,
    outputs, spread)."""
    import torch

    from paper_2609_09240_amd import tq
    launches = step_launches(mats, xs)
    dev = xs[0][0].device
    outs = [[torch.empty(m.n_out, dtype=torch.float16, device=dev) for m in ms] for ms, _ in launches]
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        chain = tq.Chain([(ms, x, ys) for (ms, x), ys in zip(launches, outs)], stream=stream)
        for _ in range(warmup):
            chain.run(stream=stream)
    torch.cuda.synchronize()
    t_start = torch.cuda.Event(enable_timing=True)
    t_stop = torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(stream):
        t_start.record(stream)
        for _ in range(steps):
            chain.run(stream=stream)
        t_stop.record(stream)
    torch.cuda.synchronize()
    ms_per_step = t_start.elapsed_time(t_stop) / steps
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    with torch.cuda.stream(stream):
        for a, b in evs:
            a.record(stream)
            chain.run(stream=stream)
            b.record(stream)
    torch.cuda.synchronize()
    per_step = sorted(a.elapsed_time(b) * 1e3 for a, b in evs)
    spread = [round(per_step[min(len(per_step) - 1, int(q / 100 * len(per_step)))], 2) for q in (10, 50, 90)]
    err = chain.error_flag()
    if err:
        raise RuntimeError("tq_gemv_chain: a stage wait gave up (sync error flag set)")
    return ms_per_step, chain, outs, spread


def algorithmic_bytes(launches):
    total = 0
    for ms, x in launches:
        for m in ms:
            total += m.nbytes() + 2 * m.n_in + 2 * m.n_out
    return total


def kernel_source_hash(path):
    """sha256[:16] of the sources of the step's dominant kernel."""
    import hashlib
    files = ("chain.hip", "gemv_decode.h") if path == "chain" else ("gemv.hip", "gemv_decode.h")
    h = hashlib.sha256()
    for f in files:
        h.update(open(os.path.join(ROOT, "paper_2609_09240_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(path):
    """HBM bytes per launch of the step's dominant kernel from the committed
    rocprofv3 counter summary, if it was taken on the current kernel sources
    (else None)."""
    import re
    name = "chain_kernel_qwen3_8b_decode_step.md" if path == "chain" else "gemv_qwen3_8b_decode_step.md"
    prof = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(prof):
        return None
    m = re.search(r"traffic_bytes_per_launch = (\d+)\s+\(sources sha256\[:16\] = ([0-9a-f]+)\)",
                  open(prof).read())
    return float(m.group(1)) if m and m.group(2) == kernel_source_hash(path) else None


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_rate(layers):
    """Algorithmic bytes and seconds of the oracle's gemv over `layers`."""
    import numpy as np

    from oracle import accounting, codec, packed
    from paper_2609_09240_amd import synth
    nbytes, secs = 0, 0.0
    for layer in range(layers):
        for name, _, _ in synth.PROJECTIONS:
            inp = synth.projection(name, layer, cfg=3)
            x = synth.stage_activations(synth.STAGE_OF[name], layer, cfg=3)
            c0, _ = codec.pack(inp.t0.reshape(-1, 128))
            c1, _ = codec.pack(inp.t1.reshape(-1, 128))
            t = time.perf_counter()
            y = packed.gemv(inp.n_out, inp.n_in, c0, inp.s0, inp.rowptr1, inp.gidx1, c1, inp.mu1, inp.s1, x)
            secs += time.perf_counter() - t
            assert np.all(np.isfinite(y))
            nbytes += accounting.gemv_bytes(inp.n_out, inp.n_in, inp.nnz1)
    return nbytes, secs


def cpu_baseline(layers=2, layers_1t=1):
    """The oracle (numpy fp64: decode, dequantise, matvec) on the first
    layers of the same stack, with numpy's BLAS on every host core and then
    on one thread."""
    from threadpoolctl import threadpool_info, threadpool_limits
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    nbytes, secs = _oracle_rate(layers)
    with threadpool_limits(limits=1):
        nb1, s1 = _oracle_rate(layers_1t)
    return {"value": round(nbytes / secs / 1e9, 6), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "sample": f"oracle gemv (decode + fp64 dequant + fp64 matvec) of layers 0..{layers - 1} "
                      f"(7 projections each, {nbytes} algorithmic bytes) in {secs:.1f} s with BLAS on "
                      f"{threads} threads; host: {os.cpu_count()} logical CPUs, {cpu_model()}",
            "one_thread": {"value": round(nb1 / s1 / 1e9, 6), "unit": "GB/s", "cores": 1,
                           "sample": f"layer 0 (7 projections, {nb1} bytes) in {s1:.1f} s"},
            "cpu_model": cpu_model(), "logical_cpus": os.cpu_count()}


def graph_time_us(calls, reps=3, back_to_back=1):
    """Median over `reps` timed regions of a HIP graph holding `calls` (a
    list of zero-argument launches), per call, in microseconds.  Each timed
    region replays the graph `back_to_back` times between one pair of
    events, as the decode step's timed region does."""
    import torch
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        for c in calls:
            c()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        for c in calls:
            c()
    torch.cuda.synchronize()
    times = []
    for _ in range(reps + 1):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(stream):
            a.record(stream)
            for _ in range(back_to_back):
                g.replay()
            b.record(stream)
        torch.cuda.synchronize()
        times.append(a.elapsed_time(b) * 1e3 / (len(calls) * back_to_back))
    return sorted(times[1:])[reps // 2]


def copies_of(mat, n):
    """n device copies of a packed linear (same values, distinct buffers), so
    that rotating over them streams from HBM."""
    import dataclasses
    out = []
    for _ in range(n):
        kw = {f.name: getattr(mat, f.name) for f in dataclasses.fields(mat)}
        for k, v in kw.items():
            if k != "rowptr1_host" and hasattr(v, "clone"):
                kw[k] = v.clone()
        out.append(type(mat)(**kw))
    return out


def paper_representation_line(dev, layers=36, steps=10, warmup=3):
    """The decode step in the paper's own representation: an offset on every
    group and 3.6% two-plane groups (section 3), same shapes and protocol."""
    import torch
    mats, xs = build_stack(layers, dev, paper_representation=True)
    ms_per_step, launches, graph, outs = time_stack(mats, xs, steps, warmup)
    step_bytes = algorithmic_bytes(launches)
    weight_bytes = sum(m.nbytes() for ms, _ in launches for m in ms)
    n_weights = sum(m.n_out * m.n_in for ms, _ in launches for m in ms)
    line = {"bench": "decode_step_paper_representation", "layers": layers, "steps": steps,
            "two_plane_fraction": 0.036, "group_offsets": "every group",
            "us_per_step": round(ms_per_step * 1e3, 2),
            "GBps": round(step_bytes / (ms_per_step * 1e-3) / 1e9, 2),
            "algorithmic_bytes_per_step": step_bytes,
            "stored_bits_per_weight": round(8 * weight_bytes / n_weights, 4)}
    del graph, outs, launches, mats, xs
    torch.cuda.empty_cache()
    return line


def graph_node_floor(dev, nodes=144, reps=5, back_to_back=10):
    """Per-node time of a HIP graph of `nodes` nearly empty launches
    (tq_validate over one group: one workgroup reading 26 bytes), timed like
    the step: the gap between graph nodes, the dispatch and one memory round
    trip.  A stage's per-launch time minus this floor is what its work adds
    to a launch that does almost nothing."""
    import torch

    from paper_2609_09240_amd import tq
    codes = torch.zeros(64, dtype=torch.uint8, device=dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    us = graph_time_us([lambda: tq.tq_validate(codes, 1, d_err=err, stream=torch.cuda.current_stream())] * nodes,
                       reps=reps, back_to_back=back_to_back)
    return {"us_per_node": round(us, 3), "nodes": nodes, "kernel": "validate_kernel over one group"}


def per_stage(mats, xs, reps=5, back_to_back=10):
    """Each stage kind of the step (q+k+v, o, gate+up, down) timed on its
    own: a HIP graph of its 36 launches (one per layer, each on that layer's
    weights, so they stream from HBM), replayed 10 times back to back
    between one pair of HIP events on the replay stream (as the step is
    timed), median of 5.  Per launch: the timed region over the launches it
    holds (it includes the gap between graph nodes, so it bounds the kernel
    duration from above)."""
    import torch

    from paper_2609_09240_amd import synth, tq
    out = {}
    for s, names in enumerate(synth.STAGES):
        launches = [([mats[layer][n] for n in names], xs[layer][s]) for layer in range(len(mats))]
        ys = [[torch.empty(m.n_out, dtype=torch.float16, device=xs[0][0].device) for m in ms] for ms, _ in launches]
        calls = []
        for (ms, x), y in zip(launches, ys):
            if len(ms) == 1:
                calls.append(lambda ms=ms, x=x, y=y: tq.tq_gemv(ms[0], x, y=y[0], stream=torch.cuda.current_stream()))
            else:
                calls.append(lambda ms=ms, x=x, y=y: tq.tq_gemv_grouped(ms, x, ys=y, stream=torch.cuda.current_stream()))
        us = graph_time_us(calls, reps=reps, back_to_back=back_to_back)
        nbytes = sum(m.nbytes() + 2 * m.n_in + 2 * m.n_out for m in launches[0][0])
        out["+".join(names)] = {"us_per_launch": round(us, 3), "bytes_per_launch": nbytes,
                                "GBps": round(nbytes / us / 1e3, 1), "frac": round(nbytes / us / 1e3 / HBM_PEAK_GBS, 4)}
    return out


def config_suite(dev, min_bytes=1 << 30, reps=5):
    """Single launches of each BASELINE-style configuration, rotating over
    enough distinct copies (>= 1 GiB) that every call streams its weights
    from HBM: the 1024 x 4096 one-plane linear, q/k/v/o, gate/up/down (MLP
    inputs with outlier channels), and tq_unpack_fp16 over the full 36-layer
    projection set.  Per call: HIP-event graph time over the calls (gaps
    included; rocprofv3 gives the kernel durations)."""
    import torch

    from paper_2609_09240_amd import synth, tq
    lines = []
    cases = [("cfg0 single linear 1024x4096", synth.single_linear()[0], synth.single_linear()[1])]
    for name in ("q", "k", "v", "o", "gate", "up", "down"):
        cfg = 1 if name in ("q", "k", "v", "o") else 2
        cases.append((f"cfg{cfg} {name}", synth.projection(name, layer=0, cfg=cfg),
                      synth.stage_activations(synth.STAGE_OF[name], layer=0, cfg=cfg)))
    for label, inp, x in cases:
        base = tq.PackedLinear.from_inputs(inp, dev)
        n = max(2, -(-min_bytes // base.nbytes()))
        mats = copies_of(base, n)
        xd = torch.from_numpy(x).to(dev)
        y = torch.empty(inp.n_out, dtype=torch.float16, device=dev)
        us = graph_time_us([lambda m=m: tq.tq_gemv(m, xd, y=y, stream=torch.cuda.current_stream()) for m in mats],
                           reps=reps)
        nbytes = base.nbytes() + 2 * inp.n_in + 2 * inp.n_out
        log(f"{label}: {us:.3f} us per call")
        lines.append({"bench": "config_cold", "config": label, "shape": f"{inp.n_out}x{inp.n_in}",
                      "two_plane_groups": inp.nnz1, "copies": n, "us_per_call": round(us, 3),
                      "bytes": nbytes, "GBps": round(nbytes / us / 1e3, 1),
                      "frac": round(nbytes / us / 1e3 / HBM_PEAK_GBS, 4)})
        del mats, base
        torch.cuda.empty_cache()
    # cfg4: tq_unpack_fp16 of every projection of the 36-layer stack, in
    # order, each into its own output (13.9 GB written, 1.7 GB read: both
    # far beyond the caches).
    mats, _ = build_stack(36, dev)
    seq = [m for layer in mats for m in layer.values()]
    outs = [torch.empty(m.n_out, m.n_in, dtype=torch.float16, device=dev) for m in seq]
    for m, w in zip(seq[:7], outs[:7]):
        tq.tq_unpack_fp16(m, w=w)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for m, w in zip(seq, outs):
        tq.tq_unpack_fp16(m, w=w)
    b.record()
    torch.cuda.synchronize()
    t_total = a.elapsed_time(b) * 1e3
    log(f"cfg4 tq_unpack_fp16: {t_total:.1f} us for {len(seq)} calls")
    nbytes = sum(m.nbytes() + 2 * m.n_out * m.n_in for m in seq)
    nw = sum(m.n_out * m.n_in for m in seq)
    lines.append({"bench": "config_cold", "config": "cfg4 tq_unpack_fp16, 36-layer set (252 matrices)",
                  "weights": nw, "us_total": round(t_total, 1), "bytes": nbytes,
                  "GBps": round(nbytes / t_total / 1e3, 1), "frac": round(nbytes / t_total / 1e3 / HBM_PEAK_GBS, 4)})
    del outs, seq, mats
    torch.cuda.empty_cache()
    return lines


def extra_suite(dev):
    """Small batch (MFMA path), codec throughput, and the paper's 4096 x 2560
    comparison (dense fp16 GEMV, packed GEMV, unpack + dense GEMV)."""
    import torch

    from paper_2609_09240_amd import synth, tq
    lines = []
    ring = 32   # copies per measurement: > 256 MB for the 12 MB matrices

    # Small batch on the MLP shapes.
    for name in ("gate", "down"):
        inp = synth.projection(name, layer=0, cfg=4)
        base = tq.PackedLinear.from_inputs(inp, dev)
        mats = copies_of(base, ring)
        for B in (1, 2, 4, 8, 16, 32, 64):
            X = torch.from_numpy(synth.stage_activations(synth.STAGE_OF[name], layer=0, cfg=4, batch=B)).to(dev)
            Y = torch.empty(B, inp.n_out, dtype=torch.float16, device=dev)
            calls = [lambda m=m: tq.tq_gemm_smallbatch(m, X, Y=Y, stream=torch.cuda.current_stream()) for m in mats]
            us = graph_time_us(calls)
            log(f"small batch {name} B={B}: {us:.2f} us per call")
            nbytes = base.nbytes() + 2 * B * (inp.n_in + inp.n_out)
            tflops = 2.0 * B * inp.n_out * inp.n_in / (us * 1e-6) / 1e12
            lines.append({"bench": "smallbatch", "matrix": f"{name} {inp.n_out}x{inp.n_in}", "batch": B,
                          "us": round(us, 2), "GBps": round(nbytes / us / 1e3, 1), "TFLOPs": round(tflops, 2),
                          "hbm_frac": round(nbytes / us / 1e3 / HBM_PEAK_GBS, 4),
                          "mfma_fp16_frac": round(tflops / 2500.0, 4)})
        del mats, base

    # Codec on the gate projection (plane 0), rotating over 6 copies (>256 MiB,
    # so each call streams from HBM rather than the last-level cache).
    inp = synth.projection("gate", layer=0, cfg=4)
    trits = [torch.from_numpy(inp.t0.reshape(-1, 128)).to(dev) for _ in range(6)]
    codes = [tq.tq_pack(t) for t in trits]
    ng = trits[0].shape[0]
    us = graph_time_us([lambda i=i: tq.tq_pack(trits[i], codes=codes[i]) for i in range(6)] * 2)
    lines.append({"bench": "tq_pack", "groups": ng, "us": round(us, 2), "GBps": round((128 + 26) * ng / us / 1e3, 1)})
    us = graph_time_us([lambda i=i: tq.tq_unpack(codes[i], ng, trits=trits[5 - i]) for i in range(6)] * 2)
    lines.append({"bench": "tq_unpack", "groups": ng, "us": round(us, 2), "GBps": round((128 + 26) * ng / us / 1e3, 1)})
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    us = graph_time_us([lambda i=i: tq.tq_validate(codes[i], ng, d_err=err) for i in range(6)] * 2)
    lines.append({"bench": "tq_validate", "groups": ng, "us": round(us, 2), "GBps": round(26 * ng / us / 1e3, 1)})
    del trits, codes
    mats = [tq.PackedLinear.from_inputs(inp, dev) for _ in range(2)]
    ws = [torch.empty(inp.n_out, inp.n_in, dtype=torch.float16, device=dev) for _ in range(3)]
    us = graph_time_us([lambda i=i: tq.tq_unpack_fp16(mats[i % 2], w=ws[i % 3]) for i in range(6)] * 2)
    nb = mats[0].nbytes() + 2 * inp.n_out * inp.n_in
    lines.append({"bench": "tq_unpack_fp16", "matrix": f"gate {inp.n_out}x{inp.n_in}", "us": round(us, 2),
                  "GBps": round(nb / us / 1e3, 1)})
    del mats, ws

    # E2M-ATQ ternarisation of a gate-sized fp16 W (12288 x 4096): the
    # one-plane ranking pass, then the pass with 10% two-plane groups.
    import numpy as np
    N, K = 12288, 4096
    W = torch.randn(N, K, device=dev, dtype=torch.float32).mul_(0.02).to(torch.float16)
    groups = W.reshape(-1, 128)
    ng = groups.shape[0]
    t0b = torch.empty((ng, 128), dtype=torch.int8, device=dev)
    s0b = torch.empty(ng, dtype=torch.float16, device=dev)
    eb = torch.empty(ng, dtype=torch.float64, device=dev)
    t_rank = graph_time_us([lambda: tq.tq_ternarize(groups, iters=0, t0=t0b, s0=s0b, energy=eb)] * 4)
    nnz = int(np.floor(0.1 * ng))
    rec_d = tq.tq_select_two_plane(eb, N, K // 128, nnz)[0]
    t1b = torch.empty((nnz, 128), dtype=torch.int8, device=dev)
    mub = torch.empty(nnz, dtype=torch.float16, device=dev)
    s1b = torch.empty(nnz, dtype=torch.float16, device=dev)
    t_fit = graph_time_us([lambda: tq.tq_ternarize(groups, rec_index=rec_d, nnz=nnz, iters=4, t0=t0b, s0=s0b,
                                                   t1=t1b, offset1=mub, scale1=s1b, want_energy=False)] * 4)
    # The same two passes with an offset on every group (one-plane groups
    # then also refine mu and s0).
    m0b = torch.empty(ng, dtype=torch.float16, device=dev)
    t_rank_off = graph_time_us([lambda: tq.tq_ternarize(groups, iters=4, t0=t0b, s0=s0b, energy=eb, offset0=m0b)]
                               * 4)
    t_fit_off = graph_time_us([lambda: tq.tq_ternarize(groups, rec_index=rec_d, nnz=nnz, iters=4, t0=t0b, s0=s0b,
                                                       t1=t1b, offset1=mub, scale1=s1b, want_energy=False,
                                                       offset0=m0b)] * 4)
    lines.append({"bench": "tq_ternarize", "matrix": f"{N}x{K} fp16", "groups": ng,
                  "rank_pass_us": round(t_rank, 2), "fit_pass_us": round(t_fit, 2), "two_plane_groups": nnz,
                  "iters": 4, "fit_pass_GBps": round(ng * (256 + 130) / t_fit / 1e3, 1),
                  "group_offsets": {"rank_pass_us": round(t_rank_off, 2), "fit_pass_us": round(t_fit_off, 2)}})
    del W, groups, t0b, s0b, eb, t1b, mub, s1b, rec_d, m0b

    # The paper's microbenchmark shape (out 4096, in 2560), cold caches.
    inp = synth.linear(4096, 2560, synth.TWO_PLANE, (9, 4096, 2560, 0))
    x = torch.from_numpy(synth.activations(2560, (9, 4096, 2560, 1))).to(dev)
    base = tq.PackedLinear.from_inputs(inp, dev)
    mats = copies_of(base, 256)
    dense = [tq.tq_unpack_fp16(m) for m in mats[:64]]
    torch.cuda.synchronize()
    y = torch.empty(4096, dtype=torch.float16, device=dev)
    t_dense = graph_time_us([lambda W=W: torch.mv(W, x, out=y) for W in dense])
    t_packed = graph_time_us([lambda m=m: tq.tq_gemv(m, x, y=y, stream=torch.cuda.current_stream()) for m in mats])
    scratch = torch.empty(4096, 2560, dtype=torch.float16, device=dev)
    t_unpack = graph_time_us([lambda m=m: (tq.tq_unpack_fp16(m, w=scratch, stream=torch.cuda.current_stream()),
                                           torch.mv(scratch, x, out=y)) for m in mats[:64]])
    lines.append({"bench": "paper_shape_4096x2560", "dense_fp16_mv_us": round(t_dense, 2),
                  "packed_gemv_us": round(t_packed, 2), "unpack_fp16_plus_mv_us": round(t_unpack, 2),
                  "packed_vs_dense": round(t_packed / t_dense, 3), "unpack_plus_mv_vs_dense": round(t_unpack / t_dense, 3),
                  "packed_bytes": base.nbytes(), "dense_bytes": 2 * 4096 * 2560})
    return lines


def stream_ceiling(nbytes, dev, reps=5):
    """Measured streaming-read ceiling at the step's byte count: tq_validate
    (a 16-byte-per-lane read-reduce kernel) over one buffer of that size,
    larger than the caches, so each pass streams from HBM."""
    import torch

    from paper_2609_09240_amd import tq
    n_groups = nbytes // 26
    buf = torch.full((26 * n_groups,), 121, dtype=torch.uint8, device=dev)   # valid codes
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        tq.tq_validate(buf, n_groups, d_err=err)
    torch.cuda.synchronize()
    times = []
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(stream):
            a.record(stream)
            tq.tq_validate(buf, n_groups, d_err=err)
            b.record(stream)
        torch.cuda.synchronize()
        times.append(a.elapsed_time(b) * 1e-3)
    assert int(err.item()) == 0
    t = sorted(times)[len(times) // 2]
    del buf
    return {"kernel": "tq_validate read-reduce over one buffer of the step's byte count",
            "bytes": 26 * n_groups, "us": round(t * 1e6, 2), "GBps": round(26 * n_groups / t / 1e9, 1)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--layers", type=int, default=36)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--configs", action="store_true",
                    help="also print one cold-cache line per configuration (single launches over >= 1 GiB of copies)")
    ap.add_argument("--extra", action="store_true",
                    help="also print small-batch, codec and 4096 x 2560 comparison lines")
    ap.add_argument("--configs-only", action="store_true",
                    help="print only the --configs lines (no decode-step line; for profiler runs)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the packed GEMV path is single-device; "
              "run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2609_09240_amd import tq
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    tq.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.configs_only:
        for line in config_suite(dev):
            print(json.dumps(line), flush=True)
        return

    mats, xs = build_stack(args.layers, dev)
    launches = step_launches(mats, xs)
    step_bytes = algorithmic_bytes(launches)
    weight_bytes = sum(m.nbytes() for ms, _ in launches for m in ms)
    n_weights = sum(m.n_out * m.n_in for ms, _ in launches for m in ms)

    # The step two ways, both timed the same way: one tq_gemv_chain launch
    # per step, and 144 launches (one per stage) in a HIP graph.  They must
    # give the same bits; `value` is the faster, named in config.workload.
    ms_chain, chain, outs_chain, spread_chain = time_chain(mats, xs, args.steps, args.warmup)
    log(f"chain: {args.steps} steps: {ms_chain * 1e3:.1f} us/step")
    ms_graph, _, graph, outs_graph = time_stack(mats, xs, args.steps, args.warmup)
    spread_graph = [time_stack.spread_us[q] for q in (10, 50, 90)]
    log(f"graph of {len(launches)} launches: {ms_graph * 1e3:.1f} us/step")
    torch.cuda.synchronize()
    for a, b in zip(outs_chain, outs_graph):
        for ya, yb in zip(a, b):
            if not torch.equal(ya.view(torch.int16), yb.view(torch.int16)):
                raise RuntimeError("chain and per-launch GEMV outputs differ")
    del chain, outs_chain, graph, outs_graph
    torch.cuda.empty_cache()
    stages = per_stage(mats, xs)
    node_floor = graph_node_floor(dev)
    for v in stages.values():
        v["us_minus_node_floor"] = round(v["us_per_launch"] - node_floor["us_per_node"], 3)
    log("per stage: " + ", ".join(f"{k} {v['us_per_launch']} us" for k, v in stages.items())
        + f"; graph node floor {node_floor['us_per_node']} us")
    use_chain = ms_chain <= ms_graph
    ms_per_step = ms_chain if use_chain else ms_graph
    spread = spread_chain if use_chain else spread_graph
    gbs = step_bytes / (ms_per_step * 1e-3) / 1e9
    paths = {
        "chain": {"us_per_step": round(ms_chain * 1e3, 2), "GBps": round(step_bytes / (ms_chain * 1e-3) / 1e9, 2),
                  "launches_per_step": 1, "kernel": "chain_kernel",
                  "what": "tq_gemv_chain: every stage in one cooperative launch"},
        "graph": {"us_per_step": round(ms_graph * 1e3, 2), "GBps": round(step_bytes / (ms_graph * 1e-3) / 1e9, 2),
                  "launches_per_step": len(launches), "kernel": "gemv_kernel",
                  "what": "one tq_gemv / tq_gemv_grouped launch per stage, captured in a HIP graph"},
    }

    # Roofline of the dominant kernel.  Chain: one launch per step, its
    # duration is the timed region.  Graph: the timed region over the
    # launches it holds (an upper bound on the kernel duration: it includes
    # the gaps between graph nodes).
    nl = 1 if use_chain else len(launches)
    avg_ms = ms_per_step / nl
    achieved = step_bytes / nl / (avg_ms * 1e-3) / 1e9

    # Calibration for HBM counters: a plain copy of known size (outside the
    # timed region), so FETCH_SIZE / WRITE_SIZE can be scaled.
    cal = torch.empty(COPY_BYTES // 2, dtype=torch.float16, device=dev)
    cal_dst = torch.empty_like(cal)
    for _ in range(3):
        cal_dst.copy_(cal)
    torch.cuda.synchronize()
    del cal, cal_dst

    ceiling = stream_ceiling(step_bytes, dev)
    log(f"streaming-read ceiling: {ceiling['GBps']:.1f} GB/s")

    result = {
        "metric": "packed ternary GEMV HBM GB/s (% of peak) + us per Qwen3-8B decode-step linears",
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 6),
        "us_per_step": round(ms_per_step * 1e3, 2),
        "step_us_p10_p50_p90": spread,
        "pct_of_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2),
        "pct_of_stream_ceiling": round(100 * gbs / ceiling["GBps"], 2),
        "stream_ceiling": ceiling,
        "step_paths": paths,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp16 activations x base-3 packed ternary weights, fp32 accumulation",
        "data": "synthetic (seeded; Qwen3-8B projection shapes, 10% two-plane groups)",
        "config": {
            "workload": f"Qwen3-8B decode-step linear stack, batch 1: {args.layers} layers x "
                        "{q,k,v,o,gate,up,down} as 144 dependent stages (q+k+v and gate+up grouped), timed as "
                        + ("one tq_gemv_chain launch per step" if use_chain else
                           "144 tq_gemv/tq_gemv_grouped launches per step in a HIP graph"),
            "step_path": "chain" if use_chain else "graph",
            "layers": args.layers,
            "stages_per_step": len(launches),
            "weights_per_step": n_weights,
            "packed_weight_bytes": weight_bytes,
            "algorithmic_bytes_per_step": step_bytes,
            "stored_bits_per_weight": round(8 * weight_bytes / n_weights, 4),
            "parallelism": "single GPU",
        },
        "roofline": {
            "bound": "hbm",
            "kernel": "chain_kernel" if use_chain else "gemv_kernel",
            "achieved": round(achieved, 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": measured_traffic("chain" if use_chain else "graph"),
            "avg_launch_us": round(avg_ms * 1e3, 3),
            "bytes_per_launch": round(step_bytes / nl, 1),
            "per_stage": stages,
            "graph_node_floor": node_floor,
            "dominant": max(stages, key=lambda k: stages[k]["us_per_launch"]),
        },
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample ...")
        result["cpu_baseline"] = cpu_baseline()
    print(json.dumps(result), flush=True)
    if args.configs or args.extra:
        del launches, mats, xs
        torch.cuda.empty_cache()
    if args.configs:
        for line in config_suite(dev):
            print(json.dumps(line), flush=True)
    if args.extra:
        print(json.dumps(paper_representation_line(dev)), flush=True)
        for line in extra_suite(dev):
            print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
