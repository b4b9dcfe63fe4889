#!/usr/bin/env python3
"""Benchmark of the RRS W4A4 linear layer on one MI355X.

A step is one pass of the whole hot path on one batch: rotate + runtime smooth
+ per-token INT4 quantization (rrs_rotate_smooth_quant) followed by the
smoothing-fused W4A4 GEMM (rrs_w4a4_gemm), i.e. exactly what rrs_linear runs.
Workload: the LLaMA-7B-shaped fused QKV projection, M=2048 tokens, K=4096,
N=12288, smoothing group 128, on seeded synthetic outlier-laden activations and
random N(0, 0.02^2) weights (offline weight preparation is outside the timed
region). Inputs are resident in HBM before timing starts.

value = 2*M*N*K / (time per step), effective TOPS of the whole step, where the
time per step is that of K back-to-back steps between one pair of HIP events.
The roofline object covers the dominant kernel (the GEMM): its average
duration is taken from HIP events recorded around it on the launch stream, in
K further steps that also give the breakdown (their per-kernel events add
their own cost to each step, reported as step_us_with_kernel_events).
A decode-shaped measurement (M=8, K=8192, N=28672) reports HBM GB/s of the
GEMM over algorithmic bytes, cycling through 4 weight copies (470 MB, more
than the 256 MB Infinity Cache) so that every call streams its weight from HBM:
back to back (one event pair around the calls, as a decode loop issues them),
and with an event after every call (*_per_call_events, gaps included).
Further objects on the same line: few-token layers at the decode shape
(M = 1..64), the gate/up and large prefill configurations against their own
rooflines, the runtime-reorder comparison, the kernel comparison of the three
scale schemes, and the CPU oracle baseline.

Prints one JSON line.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "effective W4A4 TOPS at M=2048,K=4096,N=12288; HBM GB/s at M=8 decode"
# HBM bytes per launch of the GEMM kernel on this workload, from two rocprofv3
# --pmc runs (FETCH_SIZE, WRITE_SIZE) scaled by a 256 MiB copy-kernel
# calibration (profiles/gemm_main_kernel_qkv.md), keyed by the sha1 prefix of
# the kernel source they were measured on. Any other source reports null.
GEMM_TRAFFIC_BYTES = {"a55e13cd5d24": 159.81e6}
INT8_MFMA_PEAK_TOPS = 5000.0   # MI355X dense int8 MFMA, 5.0 POP/s
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E


def gemm_traffic():
    import hashlib
    src = os.path.join(ROOT, "paper_2409_20361_amd", "csrc", "rrs_gemm.hip")
    with open(src, "rb") as f:
        sha = hashlib.sha1(f.read()).hexdigest()[:12]
    return GEMM_TRAFFIC_BYTES.get(sha)


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-decode", action="store_true", help="skip the decode measurement")
    ap.add_argument("--decode-only", action="store_true",
                    help="only the decode measurement (for per-kernel profiles)")
    ap.add_argument("--decode-steps", type=int, default=100)
    ap.add_argument("--no-tiled", action="store_true",
                    help="decode measurement on the row-major weights only")
    ap.add_argument("--no-graph", action="store_true",
                    help="skip the HIP-graph replay timings")
    ap.add_argument("--graph-only", action="store_true",
                    help="only the HIP-graph replay timings")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the gate/up and large prefill configurations")
    ap.add_argument("--configs-only", action="store_true",
                    help="only the gate/up and large prefill configurations")
    ap.add_argument("--no-reorder", action="store_true",
                    help="skip the runtime-reorder comparison")
    ap.add_argument("--reorder-only", action="store_true",
                    help="only the runtime-reorder comparison")
    ap.add_argument("--no-schemes", action="store_true",
                    help="skip the per-channel / Runtime Smooth / sub-channel kernel comparison")
    ap.add_argument("--schemes-only", action="store_true",
                    help="only the kernel comparison of the three scale schemes")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run 5 plain 256 MiB device copies, the reference kernel "
                         "for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE counters")
    return ap.parse_args()


def copy_calibration(torch):
    n = 256 << 20
    src = torch.empty(n, dtype=torch.uint8, device="cuda:0").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    log(f"copy calibration: 5 copies of {n} bytes")


def prewarm(torch, fn, seconds=0.3):
    """Run `fn` untimed for a fixed wall time before the warmup steps: the GPU
    takes tens of milliseconds of load to reach its steady clock, far longer
    than a few warmup steps of a sub-millisecond workload."""
    t0 = time.perf_counter()
    n = 0
    while time.perf_counter() - t0 < seconds:
        for _ in range(20):
            fn()
        torch.cuda.synchronize()
        n += 20
    log(f"pre-warm: {n} untimed calls in {time.perf_counter() - t0:.2f} s")


def qkv_step_bench(args, torch, rrs, synth):
    w = synth.WORKLOADS["qkv"]
    dev = torch.device("cuda:0")
    log(f"workload qkv M={w.M} K={w.K} N={w.N} g={w.g}: generating inputs")
    X = torch.from_numpy(synth.activations(w)).to(dev)
    Wq, beta = rrs.prepare_weight(torch.from_numpy(synth.weights(w)).to(dev))
    Xq = torch.empty((w.M, w.K // 2), dtype=torch.uint8, device=dev)
    a = torch.empty((w.M,), dtype=torch.float32, device=dev)
    s = torch.empty((w.G,), dtype=torch.float32, device=dev)
    Y = torch.empty((w.M, w.N), dtype=torch.float16, device=dev)
    ws = torch.zeros((rrs.workspace_bytes(w.M, w.K, w.g),), dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()

    def step(evs=None):
        if evs is not None:
            evs[0].record()
        rrs.rotate_smooth_quant(X, w.g, workspace=ws, out=(Xq, a, s))
        if evs is not None:
            evs[1].record()
        rrs.w4a4_gemm(Xq, a, s, Wq, beta, w.g, out=Y)
        if evs is not None:
            evs[2].record()

    prewarm(torch, step)
    log(f"warmup {args.warmup} steps")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # The timed region: K steps between one pair of events (no event between
    # the kernels: every event record drains the stream, which would add its
    # own cost to each step).
    e_start = torch.cuda.Event(enable_timing=True)
    e_end = torch.cuda.Event(enable_timing=True)
    log(f"timing {args.steps} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e_start.record()
    for _ in range(args.steps):
        step()
    e_end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    step_ms = e_start.elapsed_time(e_end) / args.steps
    # The breakdown: K more steps with an event pair around each kernel, for
    # the quantizer's and the GEMM's own durations (the roofline's `achieved`).
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    log(f"timing {args.steps} steps with per-kernel events")
    torch.cuda.synchronize()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    quant_ms = [e[0].elapsed_time(e[1]) for e in evs]
    gemm_ms = [e[1].elapsed_time(e[2]) for e in evs]
    step_ev_ms = evs[0][0].elapsed_time(evs[-1][2]) / args.steps
    return w, dict(step_ms=step_ms, wall_ms=wall * 1e3 / args.steps, step_ev_ms=step_ev_ms,
                   quant_ms=sum(quant_ms) / len(quant_ms), gemm_ms=sum(gemm_ms) / len(gemm_ms),
                   gemm_ms_min=min(gemm_ms), quant_ms_min=min(quant_ms),
                   gemm_ms_med=sorted(gemm_ms)[len(gemm_ms) // 2],
                   quant_ms_med=sorted(quant_ms)[len(quant_ms) // 2])


def decode_bench(args, torch, rrs, synth):
    w = synth.WORKLOADS["decode"]
    dev = torch.device("cuda:0")
    log(f"decode M={w.M} K={w.K} N={w.N}: generating inputs")
    X = torch.from_numpy(synth.activations(w)).to(dev)
    W = torch.from_numpy(synth.weights(w)).to(dev)
    Xq, a, s = rrs.rotate_smooth_quant(X, w.g)
    Y = torch.empty((w.M, w.N), dtype=torch.float16, device=dev)
    lws = torch.zeros((rrs.linear_workspace_bytes(w.M, w.K, w.g),), dtype=torch.uint8,
                      device=dev)
    alg = (w.M * w.K // 2 + 4 * w.M + 4 * w.G + w.N * w.K // 2 + 4 * w.N + 2 * w.M * w.N)
    n = args.decode_steps

    def measure(flags):
        Wq0, beta = rrs.prepare_weight(W, flags=flags)
        copies = [Wq0] + [Wq0.clone() for _ in range(3)]   # 4 x 117 MB > 256 MB MALL
        it = iter(range(1 << 30))
        prewarm(torch, lambda: rrs.w4a4_gemm(Xq, a, s, copies[next(it) % 4], beta, w.g, out=Y,
                                             flags=flags))
        torch.cuda.synchronize()

        def back_to_back(fn):
            # n calls between one event pair, as a decode loop issues them
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            for i in range(n):
                fn(i)
            e1.record()
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) / n

        def per_call(fn):
            # an event after every call: each record drains the stream, so
            # these include the gap before every launch
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
            ev[0].record()
            for i in range(n):
                fn(i)
                ev[i + 1].record()
            torch.cuda.synchronize()
            return [ev[i].elapsed_time(ev[i + 1]) for i in range(n)]

        gemm = lambda i: rrs.w4a4_gemm(Xq, a, s, copies[i % 4], beta, w.g, out=Y, flags=flags)  # noqa: E731
        lin = lambda i: rrs.linear(X, copies[i % 4], beta, w.g, workspace=lws, out=Y,  # noqa: E731
                                   flags=flags)
        gb = back_to_back(gemm)
        lb = back_to_back(lin)
        g_ms = per_call(gemm)
        l_ms = per_call(lin)
        gm = sum(g_ms) / n
        lm = sum(l_ms) / n
        return {
            "gemm_us": round(gb * 1e3, 3),
            "gemm_GBps": round(alg / (gb * 1e-3) / 1e9, 1),
            "gemm_frac_hbm": round(alg / (gb * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "linear_us": round(lb * 1e3, 3),
            "linear_GBps": round(alg / (lb * 1e-3) / 1e9, 1),
            "gemm_us_per_call_events": round(gm * 1e3, 3),
            "gemm_us_per_call_events_min": round(min(g_ms) * 1e3, 3),
            "linear_us_per_call_events": round(lm * 1e3, 3),
        }

    out = {"config": {"workload": "decode", "M": w.M, "K": w.K, "N": w.N, "group_size": w.g},
           "algorithmic_bytes": alg, "weight_copies": 4, "weight_layout": "row-major"}
    out.update(measure(0))
    if not args.no_tiled:
        out["tiled"] = measure(rrs.WEIGHT_TILED)
    return out


def graph_bench(torch, rrs, synth, reps=50):
    """The same calls replayed from a HIP graph (torch.cuda.CUDAGraph on the
    library's launches): the qkv step (quantizer + GEMM) and the decode GEMM
    and layer (4 weight copies, one captured call per copy). Replays remove
    the host launch cost and the gaps between back-to-back launches; the
    kernels and their work are unchanged."""
    dev = torch.device("cuda:0")
    out = {}

    def timed(fn_capture, per_replay):
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            fn_capture()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            fn_capture()
        prewarm(torch, graph.replay, seconds=0.2)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            graph.replay()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / (reps * per_replay)

    w = synth.WORKLOADS["qkv"]
    X = torch.from_numpy(synth.activations(w)).to(dev)
    Wq, beta = rrs.prepare_weight(torch.from_numpy(synth.weights(w)).to(dev))
    Xq = torch.empty((w.M, w.K // 2), dtype=torch.uint8, device=dev)
    a = torch.empty((w.M,), dtype=torch.float32, device=dev)
    s = torch.empty((w.G,), dtype=torch.float32, device=dev)
    Y = torch.empty((w.M, w.N), dtype=torch.float16, device=dev)
    ws = torch.zeros((rrs.workspace_bytes(w.M, w.K, w.g),), dtype=torch.uint8, device=dev)

    def step():
        rrs.rotate_smooth_quant(X, w.g, workspace=ws, out=(Xq, a, s))
        rrs.w4a4_gemm(Xq, a, s, Wq, beta, w.g, out=Y)
    step_us = timed(step, 1)
    ops = 2.0 * w.M * w.N * w.K
    out["qkv"] = {"step_us": round(step_us, 2),
                  "TOPS": round(ops / (step_us * 1e-6) / 1e12, 1)}
    del X, Wq, Xq, Y

    w = synth.WORKLOADS["decode"]
    X = torch.from_numpy(synth.activations(w)).to(dev)
    Wq0, beta = rrs.prepare_weight(torch.from_numpy(synth.weights(w)).to(dev))
    copies = [Wq0] + [Wq0.clone() for _ in range(3)]
    Xq, a, s = rrs.rotate_smooth_quant(X, w.g)
    Y = torch.empty((w.M, w.N), dtype=torch.float16, device=dev)
    lws = torch.zeros((rrs.linear_workspace_bytes(w.M, w.K, w.g),), dtype=torch.uint8,
                      device=dev)

    def gemms():
        for c in copies:
            rrs.w4a4_gemm(Xq, a, s, c, beta, w.g, out=Y)

    def linears():
        for c in copies:
            rrs.linear(X, c, beta, w.g, workspace=lws, out=Y)
    alg = (w.M * w.K // 2 + 4 * w.M + 4 * w.G + w.N * w.K // 2 + 4 * w.N + 2 * w.M * w.N)
    g_us = timed(gemms, len(copies))
    l_us = timed(linears, len(copies))
    out["decode"] = {"gemm_us": round(g_us, 2),
                     "gemm_GBps": round(alg / (g_us * 1e-6) / 1e9, 1),
                     "gemm_frac_hbm": round(alg / (g_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                     "linear_us": round(l_us, 2),
                     "linear_GBps": round(alg / (l_us * 1e-6) / 1e9, 1)}
    return out


def quant_bytes(w):
    """Algorithmic HBM bytes of rrs_rotate_smooth_quant: read X, write Xq, alpha, s."""
    return 2 * w.M * w.K + w.M * w.K // 2 + 4 * w.M + 4 * w.G


def config_bench(torch, rrs, synth, names=("gateup", "large"), reps=10):
    """The other prefill configurations, each against its own roofline: the GEMM
    (int8 MFMA peak) and the quantizer (HBM) timed alone with HIP events, and
    the whole layer."""
    dev = torch.device("cuda:0")
    out = {}
    for name in names:
        w = synth.WORKLOADS[name]
        log(f"config {name} M={w.M} K={w.K} N={w.N} g={w.g}")
        X = torch.from_numpy(synth.activations(w)).to(dev)
        W = torch.from_numpy(synth.weights(w)).to(dev)
        Wq, beta = rrs.prepare_weight(W)
        del W
        Xq = torch.empty((w.M, w.K // 2), dtype=torch.uint8, device=dev)
        a = torch.empty((w.M,), dtype=torch.float32, device=dev)
        s = torch.empty((w.G,), dtype=torch.float32, device=dev)
        Y = torch.empty((w.M, w.N), dtype=torch.float16, device=dev)
        qws = torch.zeros((rrs.workspace_bytes(w.M, w.K, w.g),), dtype=torch.uint8, device=dev)
        lws = torch.zeros((rrs.linear_workspace_bytes(w.M, w.K, w.g),), dtype=torch.uint8,
                          device=dev)
        rrs.rotate_smooth_quant(X, w.g, workspace=qws, out=(Xq, a, s))
        calls = {
            "quant": lambda: rrs.rotate_smooth_quant(X, w.g, workspace=qws, out=(Xq, a, s)),
            "gemm": lambda: rrs.w4a4_gemm(Xq, a, s, Wq, beta, w.g, out=Y),
            "linear": lambda: rrs.linear(X, Wq, beta, w.g, workspace=lws, out=Y),
        }
        row = {"M": w.M, "K": w.K, "N": w.N, "group_size": w.g}
        for key, fn in calls.items():
            prewarm(torch, fn, seconds=0.2)
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
            ev[0].record()
            for i in range(reps):
                fn()
                ev[i + 1].record()
            torch.cuda.synchronize()
            t = sorted(ev[i].elapsed_time(ev[i + 1]) * 1e3 for i in range(reps))
            row[key + "_us"] = round(sum(t) / reps, 2)
            row[key + "_us_median"] = round(t[reps // 2], 2)
        ops = 2.0 * w.M * w.N * w.K
        row["gemm_TOPS"] = round(ops / (row["gemm_us"] * 1e-6) / 1e12, 1)
        row["gemm_frac_int8_peak"] = round(row["gemm_TOPS"] / INT8_MFMA_PEAK_TOPS, 4)
        row["linear_TOPS"] = round(ops / (row["linear_us"] * 1e-6) / 1e12, 1)
        qb = quant_bytes(w)
        row["quant_GBps"] = round(qb / (row["quant_us"] * 1e-6) / 1e9, 1)
        row["quant_frac_hbm"] = round(row["quant_GBps"] / HBM_PEAK_GBS, 4)
        out[name] = row
        del X, Wq, Y, Xq, lws
        torch.cuda.empty_cache()
    return out


def few_token_bench(torch, rrs, synth, reps=50):
    """Few-token layers at the decode shape (K=8192, N=28672, g=128) for
    M = 1, 2, 4, 8, 16, 32, 64: quantizer, GEMM and the whole layer, each timed
    with HIP events around 50 back-to-back calls, weights cycling through 4
    copies. At M = 1 and 2 the layer is one launch (every workgroup of the
    GEMM quantizes the rows itself); otherwise the quantizer is one launch
    with one workgroup per row and the GEMM the weight-streaming kernel up to
    M = 32 (eight waves from 17 tokens) or the few-token kernel at M = 64.
    The *_tiled entries
    run the same calls on the tiled weight layout."""
    dev = torch.device("cuda:0")
    base = synth.WORKLOADS["decode"]
    W = torch.from_numpy(synth.weights(base)).to(dev)
    Wq0, beta = rrs.prepare_weight(W)
    Wt0, _ = rrs.prepare_weight(W, flags=rrs.WEIGHT_TILED)
    del W
    copies = [Wq0] + [Wq0.clone() for _ in range(3)]
    tiled = [Wt0] + [Wt0.clone() for _ in range(3)]
    T = rrs.WEIGHT_TILED
    rows = []
    for M in (1, 2, 4, 8, 16, 32, 64):
        w = synth.custom("d", M, base.K, base.N, base.g, 40 + M, n_chan=82, n_spike=2,
                         spike_mag=(100, 500))
        X = torch.from_numpy(synth.activations(w)).to(dev)
        Xq = torch.empty((M, w.K // 2), dtype=torch.uint8, device=dev)
        a = torch.empty((M,), dtype=torch.float32, device=dev)
        s = torch.empty((w.G,), dtype=torch.float32, device=dev)
        Y = torch.empty((M, w.N), dtype=torch.float16, device=dev)
        qws = torch.zeros((rrs.workspace_bytes(M, w.K, w.g),), dtype=torch.uint8, device=dev)
        lws = torch.zeros((rrs.linear_workspace_bytes(M, w.K, w.g),), dtype=torch.uint8,
                          device=dev)
        rrs.rotate_smooth_quant(X, w.g, workspace=qws, out=(Xq, a, s))
        calls = {
            "quant": lambda i: rrs.rotate_smooth_quant(X, w.g, workspace=qws, out=(Xq, a, s)),
            "gemm": lambda i: rrs.w4a4_gemm(Xq, a, s, copies[i % 4], beta, w.g, out=Y),
            "linear": lambda i: rrs.linear(X, copies[i % 4], beta, w.g, workspace=lws, out=Y),
            "gemm_tiled": lambda i: rrs.w4a4_gemm(Xq, a, s, tiled[i % 4], beta, w.g, out=Y,
                                                  flags=T),
            "linear_tiled": lambda i: rrs.linear(X, tiled[i % 4], beta, w.g, workspace=lws,
                                                 out=Y, flags=T),
        }
        row = {"M": M}
        for key, fn in calls.items():
            it = iter(range(1 << 30))
            prewarm(torch, lambda: fn(next(it)), seconds=0.1)
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            for i in range(reps):
                fn(i)
            e1.record()
            torch.cuda.synchronize()
            row[key + "_us"] = round(e0.elapsed_time(e1) * 1e3 / reps, 2)
        alg = M * w.K // 2 + 4 * M + 4 * w.G + w.N * w.K // 2 + 4 * w.N + 2 * M * w.N
        row["linear_GBps"] = round(alg / (row["linear_us"] * 1e-6) / 1e9, 1)
        row["gemm_GBps"] = round(alg / (row["gemm_us"] * 1e-6) / 1e9, 1)
        row["gemm_tiled_GBps"] = round(alg / (row["gemm_tiled_us"] * 1e-6) / 1e9, 1)
        rows.append(row)
    return {"K": base.K, "N": base.N, "group_size": base.g, "weight_copies": 4, "rows": rows}


def scheme_bench(torch, rrs, reps=30):
    """Kernel comparison of Section 4.5 (Fig. 6): per-channel, Runtime Smooth and
    sub-channel A4W4 on the shared 128 x 128 skeleton, plus the tuned Runtime Smooth
    kernel, at LLaMA-7B shapes (hidden 4096, sequence length 1024, 1/2/4 sequences).
    The GEMMs only read codes and scales, so they run on random packed codes and
    positive scales generated on the GPU."""
    dev = torch.device("cuda:0")
    g = 128
    K = 4096
    G = K // g
    gen = torch.Generator(device=dev).manual_seed(7)
    rows = []
    for N, proj in ((4096, "o_proj"), (12288, "qkv_proj"), (22016, "gate_up_proj")):
        Wq = torch.randint(0, 256, (N, K // 2), dtype=torch.uint8, device=dev, generator=gen)
        wN = torch.rand((N,), device=dev, generator=gen) + 0.5
        wGN = torch.rand((G, N), device=dev, generator=gen) + 0.5
        for M in (1024, 2048, 4096):
            Xq = torch.randint(0, 256, (M, K // 2), dtype=torch.uint8, device=dev, generator=gen)
            aM = torch.rand((M,), device=dev, generator=gen) + 0.5
            aGM = torch.rand((G, M), device=dev, generator=gen) + 0.5
            s = torch.rand((G,), device=dev, generator=gen) + 0.5
            Y = torch.empty((M, N), dtype=torch.float16, device=dev)
            calls = {
                "per_channel": lambda: rrs.w4a4_gemm_scheme(rrs.SCHEME_PER_CHANNEL, Xq, aM, None,
                                                            Wq, wN, g, out=Y),
                "runtime_smooth": lambda: rrs.w4a4_gemm_scheme(rrs.SCHEME_RUNTIME_SMOOTH, Xq, aM,
                                                               s, Wq, wN, g, out=Y),
                "sub_channel": lambda: rrs.w4a4_gemm_scheme(rrs.SCHEME_SUB_CHANNEL, Xq, aGM,
                                                            None, Wq, wGN, g, out=Y),
                "rrs_tuned": lambda: rrs.w4a4_gemm(Xq, aM, s, Wq, wN, g, out=Y),
                "per_channel_tuned": lambda: rrs.w4a4_gemm_per_channel(Xq, aM, Wq, wN, out=Y),
            }
            row = {"proj": proj, "M": M, "N": N, "K": K}
            for name, fn in calls.items():
                for _ in range(5):
                    fn()
                torch.cuda.synchronize()
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record()
                for _ in range(reps):
                    fn()
                e1.record()
                torch.cuda.synchronize()
                row[name + "_us"] = round(e0.elapsed_time(e1) * 1e3 / reps, 2)
            pc = row["per_channel_us"]
            row["rs_overhead"] = round(row["runtime_smooth_us"] / pc - 1.0, 4)
            row["sub_channel_overhead"] = round(row["sub_channel_us"] / pc - 1.0, 4)
            row["tuned_rs_overhead"] = round(row["rrs_tuned_us"] / row["per_channel_tuned_us"]
                                             - 1.0, 4)
            rows.append(row)
    return {"skeleton": "128x128 tiles, i8 MFMA (per_channel, runtime_smooth, sub_channel); "
                        "tuned: the 256x128 main kernel (rrs_tuned, per_channel_tuned)",
            "group_size": g, "rows": rows}


def reorder_bench(torch, rrs, synth, reps=50):
    """Runtime channel reorder (Fig. 4 step (1) at run time) against the same
    layer without it, at the prefill (qkv) and decode shapes: quantizer,
    GEMM and the whole layer, each timed alone with HIP events. The decode
    GEMMs cycle through 4 weight copies, as in decode_bench."""
    dev = torch.device("cuda:0")
    out = {"block": rrs.REORDER_BLOCK}
    for name in ("qkv", "decode"):
        w = synth.WORKLOADS[name]
        log(f"reorder: {name} M={w.M} K={w.K} N={w.N}")
        X = torch.from_numpy(synth.activations(w)).to(dev)
        Wq0, beta = rrs.prepare_weight(torch.from_numpy(synth.weights(w)).to(dev))
        copies = [Wq0] + ([Wq0.clone() for _ in range(3)] if name == "decode" else [])
        nc = len(copies)
        Xq = torch.empty((w.M, w.K // 2), dtype=torch.uint8, device=dev)
        a = torch.empty((w.M,), dtype=torch.float32, device=dev)
        s = torch.empty((w.G,), dtype=torch.float32, device=dev)
        Xq2, a2, s2 = torch.empty_like(Xq), torch.empty_like(a), torch.empty_like(s)
        bo = torch.empty((w.K // rrs.REORDER_BLOCK,), dtype=torch.int32, device=dev)
        Y = torch.empty((w.M, w.N), dtype=torch.float16, device=dev)
        qws = torch.zeros((rrs.workspace_bytes(w.M, w.K, w.g),), dtype=torch.uint8, device=dev)
        rws = torch.zeros((rrs.reorder_workspace_bytes(w.M, w.K, w.g),), dtype=torch.uint8,
                          device=dev)
        lws = torch.zeros((rrs.linear_workspace_bytes(w.M, w.K, w.g),), dtype=torch.uint8,
                          device=dev)
        lrws = torch.zeros((rrs.linear_reorder_workspace_bytes(w.M, w.K, w.g),),
                           dtype=torch.uint8, device=dev)
        rrs.rotate_smooth_quant(X, w.g, workspace=qws, out=(Xq, a, s))
        rrs.rotate_smooth_quant_reorder(X, w.g, workspace=rws, out=(Xq2, a2, s2, bo))
        calls = {
            "quant": lambda i: rrs.rotate_smooth_quant(X, w.g, workspace=qws, out=(Xq, a, s)),
            "quant_reorder": lambda i: rrs.rotate_smooth_quant_reorder(
                X, w.g, workspace=rws, out=(Xq2, a2, s2, bo)),
            "gemm": lambda i: rrs.w4a4_gemm(Xq, a, s, copies[i % nc], beta, w.g, out=Y),
            "gemm_reorder": lambda i: rrs.w4a4_gemm_reorder(Xq2, a2, s2, copies[i % nc], beta,
                                                            bo, w.g, out=Y),
            "linear": lambda i: rrs.linear(X, copies[i % nc], beta, w.g, workspace=lws, out=Y),
            "linear_reorder": lambda i: rrs.linear_reorder(X, copies[i % nc], beta, w.g,
                                                           workspace=lrws, out=Y),
        }
        row = {"M": w.M, "K": w.K, "N": w.N, "group_size": w.g}
        for key, fn in calls.items():
            it = iter(range(1 << 30))
            prewarm(torch, lambda: fn(next(it)), seconds=0.2)
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            for i in range(reps):
                fn(i)
            e1.record()
            torch.cuda.synchronize()
            row[key + "_us"] = round(e0.elapsed_time(e1) * 1e3 / reps, 2)
        for key in ("quant", "gemm", "linear"):
            row[key + "_overhead"] = round(row[key + "_reorder_us"] / row[key + "_us"] - 1.0, 4)
        out[name] = row
        del X, Wq0, copies
    return out


def cpu_baseline(synth):
    """The CPU oracle as it stands, on a bounded sample of the same workload."""
    import numpy as np
    from oracle import rrs_oracle as O
    try:
        from threadpoolctl import threadpool_info
        cores = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        cores = os.cpu_count() or 1
    w = synth.WORKLOADS["qkv"]
    X = synth.activations(w)
    W = synth.weights(w)
    wq = O.prepare_weight(W)          # offline, not timed
    chunk = 256
    times, tq, tg = [], [], []
    for rep in range(3):
        t0 = time.perf_counter()
        act = O.rotate_smooth_quant(X, w.g)
        t1 = time.perf_counter()
        for r0 in range(0, w.M, chunk):
            P = O.group_partials(act.q[r0:r0 + chunk], wq.q, w.g)
            O.output(P, act.s, act.alpha[r0:r0 + chunk], wq.beta, norm=w.K)
        t2 = time.perf_counter()
        times.append(t2 - t0)
        tq.append(t1 - t0)
        tg.append(t2 - t1)
        if sum(times) > 20.0:
            break
    t_step = sorted(times)[len(times) // 2]
    ops = 2.0 * w.M * w.N * w.K
    return {
        "value": round(ops / t_step / 1e12, 6),
        "unit": "TOPS",
        "cores": int(cores),
        "kind": "oracle",
        "quant_s": round(sorted(tq)[len(tq) // 2], 3),
        "gemm_s": round(sorted(tg)[len(tg) // 2], 3),
        "sample": (f"the whole step on the qkv workload (all {w.M} tokens x {w.N} outputs; "
                   f"GEMM and epilogue in {chunk}-token chunks), median of {len(times)} "
                   f"run(s): {t_step:.2f} s per step; weight preparation excluded"),
    }


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "the benchmark measures one GPU (one process, no collectives); --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import torch
    import paper_2409_20361_amd as rrs
    import synth

    if not torch.cuda.is_available():
        sys.exit("bench.py needs a GPU")
    rrs.lib()
    if args.copy_calibration:
        copy_calibration(torch)
    if args.schemes_only:
        print(json.dumps({"metric": METRIC, "scheme_comparison": scheme_bench(torch, rrs)}),
              flush=True)
        return
    if args.graph_only:
        print(json.dumps({"metric": METRIC, "graph": graph_bench(torch, rrs, synth)}),
              flush=True)
        return
    if args.configs_only:
        print(json.dumps({"metric": METRIC, "configs": config_bench(torch, rrs, synth)}),
              flush=True)
        return
    if args.reorder_only:
        print(json.dumps({"metric": METRIC, "reorder": reorder_bench(torch, rrs, synth)}),
              flush=True)
        return
    if args.decode_only:
        print(json.dumps({"metric": METRIC, "decode": decode_bench(args, torch, rrs, synth),
                          "few_token": few_token_bench(torch, rrs, synth)}), flush=True)
        return
    w, r = qkv_step_bench(args, torch, rrs, synth)
    ops = 2.0 * w.M * w.N * w.K
    value = ops / (r["step_ms"] * 1e-3) / 1e12
    gemm_tops = ops / (r["gemm_ms"] * 1e-3) / 1e12
    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(r["step_ms"], 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int4",
        "data": "synthetic",
        "config": {"workload": "qkv", "M": w.M, "K": w.K, "N": w.N, "group_size": w.g,
                   "step": "rrs_rotate_smooth_quant + rrs_w4a4_gemm"},
        "roofline": {
            "bound": "mfma",
            "kernel": "gemm_main_kernel<4,false,false,false,false> (rrs_w4a4_gemm)",
            "achieved": round(gemm_tops, 2),
            "peak": INT8_MFMA_PEAK_TOPS,
            "unit": "TOP/s",
            "frac": round(gemm_tops / INT8_MFMA_PEAK_TOPS, 4),
            "traffic": gemm_traffic(),
        },
        "breakdown": {
            "quant_us": round(r["quant_ms"] * 1e3, 2),
            "gemm_us": round(r["gemm_ms"] * 1e3, 2),
            "gemm_us_min": round(r["gemm_ms_min"] * 1e3, 2),
            "gemm_us_median": round(r["gemm_ms_med"] * 1e3, 2),
            "quant_us_median": round(r["quant_ms_med"] * 1e3, 2),
            "quant_bytes": quant_bytes(w),
            "quant_GBps": round(quant_bytes(w) / (r["quant_ms"] * 1e-3) / 1e9, 1),
            "quant_frac_hbm": round(quant_bytes(w) / (r["quant_ms"] * 1e-3) / 1e9
                                    / HBM_PEAK_GBS, 4),
            "wall_ms_per_step": round(r["wall_ms"], 5),
            "step_us_with_kernel_events": round(r["step_ev_ms"] * 1e3, 2),
        },
    }
    if not args.no_decode:
        out["decode"] = decode_bench(args, torch, rrs, synth)
    if not args.no_graph:
        log("the same calls replayed from HIP graphs")
        out["graph"] = graph_bench(torch, rrs, synth)
    if not args.no_decode:
        log("few-token layers at the decode shape")
        out["few_token"] = few_token_bench(torch, rrs, synth)
    if not args.no_configs:
        out["configs"] = config_bench(torch, rrs, synth)
    if not args.no_reorder:
        out["reorder"] = reorder_bench(torch, rrs, synth)
    if not args.no_schemes:
        log("kernel comparison of the scale schemes")
        out["scheme_comparison"] = scheme_bench(torch, rrs)
    if not args.no_cpu:
        log("timing the CPU oracle baseline")
        out["cpu_baseline"] = cpu_baseline(synth)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
