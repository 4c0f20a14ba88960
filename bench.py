#!/usr/bin/env python3
"""Benchmark the GraphLeap graph-convolution hot path on one MI355X.

A step is one pass of the whole hot path over one batch: an L-block GraphLeap
stack (bootstrap kNN build, then per block the kNN build of the next graph
running concurrently with the MRConv update of this block), enqueued natively
by gl_graphleap_stack.  The default schedule puts both in one launch per block
(GL_SCHED_LOOKAHEAD_FUSED); the two-stream lookahead and the standard serial
ViG schedule run the same kernels and are timed beside it for context.  Default workload: ViG-Ti shaped,
12 blocks, B=32 images of 14x14 patches, C=192, k=9, dilation ceil(l/4),
bf16 storage with fp32 accumulation, synthetic seeded inputs already in HBM.

Prints one JSON line (rank 0): value = layers/s for the whole batch, plus the
roofline of the dominant kernel (durations measured live with HIP events on
the stream each kernel runs on) and the CPU oracle's rate on a bounded sample.

    python bench.py [--steps K] [--warmup W] [--workload vig_ti]
    python bench.py --only knn|mrconv|stack --steps K   (for profiler runs)
    python bench.py --only copy                          (HBM counter calibration)
    python bench.py --only full --steps K                (full-block stack, for profiler runs)

After the headline, the full GraphLeap ViG block (FC1, leap-ahead graph,
MRConv, FC2 + residual, FFN + residual; gl_vig_stack) is timed on the same
workload and reported under "full_block", with its own oracle sample.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "ViG graph-conv layers/sec at ViG-Ti B=32; Gram MFMA util %; gather HBM GB/s"
PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}   # dense MFMA peaks (MI355X)
PEAK_HBM_GBS = 8000.0

DESCR = {
    "vig_ti": "ViG-Ti isotropic stack: 12 GraphLeap blocks, B=32, 14x14 patches (N=196), C=192, "
              "k=9, dilation ceil(l/4); kNN graph + MRConv (FC 384->192) per block",
    "vig_b": "ViG-B isotropic stack: 16 blocks, B=64, N=196, C=640, k=9, dilation 1..4",
    "pyr_s1": "Pyramid stage 1: 2 blocks, B=32, 56x56 (N=3136), C=80, keys pooled 4x4 -> 196, k=9",
    "pyr_s2": "Pyramid stage 2: 2 blocks, B=32, 28x28 (N=784), C=160, keys pooled 2x2 -> 196, k=9",
    "hires": "High-res stress: 4 blocks, B=8, 56x56 (N=3136), C=96, full N x N kNN, k=16, d=2",
    "single": "Single isotropic layer: B=1, N=196, C=192, fp32, k=9, d=1",
    "vig_ti_448": "ViG-Ti at 448x448 input: 12 blocks, B=32, 28x28 patches (N=784), C=192, k=9, "
                  "dilation ceil(l/4)",
    "vig_s": "ViG-S isotropic stack: 12 blocks, B=32, N=196, C=320, k=9, dilation ceil(l/4)",
    "pyr_s3": "Pyramid stage 3: 6 blocks, B=32, 14x14 (N=196), C=400, k=9, d=1",
    "pyr_s4": "Pyramid stage 4: 2 blocks, B=32, 7x7 (N=49), C=640, k=9, d=1",
}


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def _code_only(src: str) -> str:
    """C++ source with its // and /* */ comments removed (string and character
    literals kept as they are)."""
    out, i, n = [], 0, len(src)
    while i < n:
        c = src[i]
        if c in "\"'":
            j = i + 1
            while j < n and src[j] != c:
                j += 2 if src[j] == "\\" else 1
            out.append(src[i:j + 1])
            i = j + 1
        elif src.startswith("//", i):
            j = src.find("\n", i)
            i = n if j < 0 else j
        elif src.startswith("/*", i):
            j = src.find("*/", i + 2)
            i = n if j < 0 else j + 2
        else:
            out.append(c)
            i += 1
    return "".join(out)


def kernel_source_sha() -> str:
    """Hash of the kernel sources' code: comments removed and whitespace runs
    collapsed, so an edit of comments or layout does not retire measurements
    taken on the same code."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2604_21290_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, f), encoding="utf-8") as fh:
            h.update(f.encode() + " ".join(_code_only(fh.read()).split()).encode())
    return h.hexdigest()[:16]


def load_traffic(kernel: str, workload: str):
    """HBM bytes per launch from a committed rocprofv3 --pmc summary, only if it
    was taken on the current kernel sources."""
    p = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(p):
        return None
    with open(p) as f:
        t = json.load(f)
    if t.get("source_sha") != kernel_source_sha():
        return None
    return t.get("bytes_per_launch")


def algorithmic(w, es):
    """Per-launch algorithmic work (bytes counted once, at their HBM size)."""
    B, N, M, C, k = w.B, w.N, w.M, w.C, w.k
    knn_flops = 2.0 * B * N * M * C
    knn_bytes = B * N * C * es + (B * M * C * es if w.pool_r > 1 else 0) + B * N * k * 4
    mr_flops = 2.0 * B * N * (2 * C) * C
    mr_bytes = (B * N * C * es                                   # x read
                + (B * M * C * es if w.pool_r > 1 else 0)        # pooled keys read
                + B * N * k * 4                                  # idx read
                + C * 2 * C * es                                 # W read
                + B * N * C * es)                                # out write
    return knn_flops, knn_bytes, mr_flops, mr_bytes


def layer_work(w, es):
    """Algorithmic work of one layer (one kNN build + one MRConv update), with
    bytes counted once each at their HBM size: X read by the build, X (and
    pooled keys) read by the update, the graph written by the build and read
    by the update, W, the output, and the key pooling's own I/O."""
    B, N, M, C, k = w.B, w.N, w.M, w.C, w.k
    pooled = w.pool_r > 1
    x = B * N * C * es
    keys = B * M * C * es if pooled else 0
    idx = B * N * k * 4
    flops = 2.0 * B * N * M * C + 2.0 * B * N * (2 * C) * C
    by = (x + keys) + (x + keys) + 2 * idx + 2 * C * C * es + x + ((x + keys) if pooled else 0)
    return flops, by


def _oracle_stack_worker(task) -> float:
    """One process of the CPU baseline: the oracle's stack on a slice of the
    batch, `reps` times, on one thread; returns its seconds."""
    x, Ws, bs, dilations, k, H, W, pool_r, reps = task
    from threadpoolctl import threadpool_limits

    import oracle as O
    with threadpool_limits(1):
        t0 = time.perf_counter()
        for _ in range(reps):
            O.stack_ref(x, Ws, bs, dilations, k, H, W, pool_r)
        return time.perf_counter() - t0


def cpu_baseline(w, images: int, min_seconds: float = 10.0) -> dict:
    """The oracle's stack on `images` of the batch, the images split over
    single-thread worker processes (one per host core, at most 16), repeated
    until at least `min_seconds` of CPU work have been timed; the rate is
    taken from the wall clock."""
    import multiprocessing
    from concurrent.futures import ProcessPoolExecutor

    import numpy as np

    from paper_2604_21290_amd import inputs as I

    S = min(images, w.B)
    ws = I.with_batch(w, S)
    x = I.make_features(ws).value
    Ws = [I.make_weight(ws, l).value for l in range(w.L)]
    bs = [I.make_bias(ws, l).value for l in range(w.L)]
    P = max(1, min(16, len(os.sched_getaffinity(0)), S))
    parts = [p for p in np.array_split(np.arange(S), P) if len(p)]
    tasks = lambda reps: [(x[p], Ws, bs, list(w.dilations), w.k, w.H, w.W, w.pool_r, reps) for p in parts]
    with ProcessPoolExecutor(len(parts), mp_context=multiprocessing.get_context("spawn")) as ex:
        # untimed: worker start-up and imports; its CPU seconds size the timed run
        first = sum(ex.map(_oracle_stack_worker, tasks(1)))
        reps = max(1, int(np.ceil(min_seconds / first)))
        t0 = time.perf_counter()
        busy = sum(ex.map(_oracle_stack_worker, tasks(reps)))
        wall = time.perf_counter() - t0
    scale = w.B / S
    return {"value": w.L * reps / (wall * scale), "unit": "layers/s", "cores": len(parts),
            "kind": "oracle",
            "sample": f"oracle.stack_ref (fp64 numpy, lookahead schedule) on {S} of {w.B} images "
                      f"for all {w.L} blocks, split by image over {len(parts)} single-thread "
                      f"processes; {reps} run(s), {wall:.2f} s wall, {busy:.1f} s of CPU work"
                      + (f"; time scaled x{scale:g} to the full batch" if scale != 1 else "")}


def cpu_full_block(w, images: int, blocks: int) -> dict:
    from threadpoolctl import threadpool_limits

    import oracle as O
    from paper_2604_21290_amd import inputs as I

    S = min(images, w.B)
    ws = I.with_batch(w, S)
    x = I.make_features(ws)
    ps = [{n: v.value for n, v in I.make_vig_params(ws, l).items()} for l in range(blocks)]
    with threadpool_limits(1):
        t0 = time.perf_counter()
        O.vig_stack_ref(x.value, ps, w.dilations[:blocks], w.k, H=w.H, W=w.W, pool_r=w.pool_r)
        dt = time.perf_counter() - t0
    scale = w.B / S
    return {"value": blocks / (dt * scale), "unit": "layers/s", "cores": 1, "kind": "oracle",
            "sample": f"oracle.vig_stack_ref (fp64, lookahead, 1 thread) on {S} of {w.B} "
                      f"images for {blocks} blocks in {dt:.2f} s; scaled x{scale:g}"}


def graph_replay(args, w, api, torch, x0, Wd, bd, dil, ws, out):
    """The fused-schedule step captured once in a HIP graph (one stream) and
    replayed; each replay is checked against the eager result first."""
    s = torch.cuda.Stream()
    lag = api.Lookahead(s, s)
    ref = torch.empty_like(out)

    def step(o):
        lag.stack(x0, w.H, w.W, Wd, bd, dil, w.k, w.pool_r, schedule=api.GL_SCHED_LOOKAHEAD_FUSED,
                  ws=ws, x_out=o)

    with torch.cuda.stream(s):
        step(ref)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    gout = torch.empty_like(out)
    with torch.cuda.graph(g, stream=s):
        step(gout)
    for _ in range(3):
        gout.zero_()
        with torch.cuda.stream(s):
            g.replay()
        torch.cuda.synchronize()
        if not torch.equal(gout, ref):
            log("graph replay differs from the eager stack; not reported")
            lag.close()
            return None
    n = max(10, args.steps // 4)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):       # replay() launches on the current stream
        e0.record(s)
        for _ in range(n):
            g.replay()
        e1.record(s)
    torch.cuda.synchronize()
    m = e0.elapsed_time(e1) / n
    lag.close()
    return {"ms_per_step": m, "layers_per_s": w.L / (m / 1e3)}


def heads_update(args, w, api, torch, x0, idx, Wdense, H=16) -> dict | None:
    """The multi-head MRConv update (gl_mrconv_heads: H heads, per-head weights
    Wh [H, hd, 2hd]) against the dense update (gl_mrconv, [C, 2C]) of the same
    layer, each averaged over launches timed with HIP events."""
    if w.C % H or w.pool_r > 1:
        return None
    hd = w.C // H
    Wh = torch.stack([torch.cat([Wdense[h * hd:(h + 1) * hd, h * hd:(h + 1) * hd],
                                 Wdense[h * hd:(h + 1) * hd, w.C + h * hd:w.C + (h + 1) * hd]], 1)
                      for h in range(H)]).contiguous()
    out = torch.empty_like(x0)
    mws = api.mrconv_workspace(w.B, w.N, w.C, w.k, w.C, x0.dtype, x0.device)
    hws = api.mrconv_heads_workspace(w.B, w.N, w.C, w.k, H, x0.dtype, x0.device)
    res = {"heads": H, "hd": hd, "weights_bytes": {"dense": Wdense.numel() * Wdense.element_size(),
                                                   "heads": Wh.numel() * Wh.element_size()}}
    n = max(20, args.steps // 4)
    calls = (("dense_us", lambda: api.mrconv(x0, idx, Wdense, out=out, ws=mws)),
             ("heads_us", lambda: api.mrconv_heads(x0, idx, Wh, out=out, ws=hws)))
    for name, fn in calls:
        for _ in range(3):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(n):
            fn()
        e1.record()
        torch.cuda.synchronize()
        res[name] = e0.elapsed_time(e1) / n * 1e3
    return res


# ViG-Py-S stage widths: the projection that follows each stage boundary
NEXT_STAGE_WIDTH = {80: 160, 160: 400, 400: 640}


def stage_transition(w, api, torch, x0, es: int, reps: int = 50) -> dict | None:
    """The stage boundary after a pyramid stage: 2 x 2 max pooling of the node
    grid (HBM-bound: the grid read once, a quarter of it written) and the
    width projection on the pooled nodes (gl_linear), each timed with HIP
    events on the stream its launches go to."""
    Cn = NEXT_STAGE_WIDTH.get(w.C)
    if w.pool_r <= 1 or Cn is None or w.H % 2 or w.W % 2:
        return None
    s = torch.cuda.current_stream()
    pooled = torch.empty((w.B, (w.H // 2) * (w.W // 2), w.C), dtype=x0.dtype, device=x0.device)
    g = torch.Generator(device=x0.device).manual_seed(5)
    Wp = (torch.rand((Cn, w.C), generator=g, device=x0.device) * 0.2 - 0.1).to(x0.dtype)
    bp = torch.zeros(Cn, dtype=x0.dtype, device=x0.device)
    y = torch.empty((w.B, pooled.shape[1], Cn), dtype=x0.dtype, device=x0.device)

    def timed(fn) -> float:
        for _ in range(5):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(s)
        for _ in range(reps):
            fn()
        e1.record(s)
        e1.synchronize()
        return e0.elapsed_time(e1) / reps * 1e-3

    t_pool = timed(lambda: api.max_pool_nodes(x0, w.H, w.W, 2, out=pooled, stream=s))
    t_proj = timed(lambda: api.linear(pooled, Wp, bp, out=y, stream=s))
    pool_bytes = (w.B * w.N * w.C + pooled.numel()) * es
    proj_flops = 2 * pooled.shape[0] * pooled.shape[1] * w.C * Cn
    return {"grid": f"{w.H}x{w.W} -> {w.H // 2}x{w.W // 2}", "width": f"{w.C} -> {Cn}",
            "max_pool_us": t_pool * 1e6, "max_pool_hbm_gbs": pool_bytes / t_pool / 1e9,
            "max_pool_hbm_frac": pool_bytes / t_pool / 1e9 / PEAK_HBM_GBS,
            "projection_us": t_proj * 1e6, "projection_tflops": proj_flops / t_proj / 1e12}


def step_percentiles(torch, step, stream, n: int) -> dict:
    """Per-stack times: one event pair per step on the stream that ends it."""
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
    torch.cuda.synchronize()
    ev[0].record(stream)
    for i in range(n):
        step()
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    import numpy as np
    t = np.array([ev[i].elapsed_time(ev[i + 1]) * 1e3 for i in range(n)])
    return {"n": n, "median_us": float(np.median(t)), "p10_us": float(np.percentile(t, 10)),
            "p90_us": float(np.percentile(t, 90))}


def cold_gather(w, api, torch, x0, idx, W, b, out, mr_bytes, reps: int = 20) -> dict:
    """The MRConv update warm and cold.  Warm: `reps` launches back to back,
    so the queue never drains.  Cold: a 512 MiB write before the launch evicts
    L2 and the 256 MB Infinity Cache; the launch is queued behind the write, and
    its time is the median of (write + update) minus the median of the write alone."""
    import numpy as np
    keys = api.pool_keys(x0, w.H, w.W, w.pool_r) if w.pool_r > 1 else None
    mws = api.mrconv_workspace(w.B, w.N, w.C, w.k, w.C, x0.dtype, x0.device)
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    s = torch.cuda.current_stream()

    def timed(fn) -> float:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(s)
        fn()
        e1.record(s)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3

    def upd():
        api.mrconv(x0, idx, W, b, keys=keys, out=out, ws=mws)

    def many():
        for _ in range(reps):
            upd()

    timed(many)
    warm = timed(many) / reps
    pair, alone = [], []
    for i in range(reps):
        pair.append(timed(lambda: (flush.fill_(i & 0xFF), upd())))
        alone.append(timed(lambda: flush.fill_((i + 1) & 0xFF)))
    cold = float(np.median(pair) - np.median(alone))
    del flush
    return {"warm_us": warm, "cold_us": cold, "hbm_gbs_warm": mr_bytes / warm / 1e3,
            "hbm_gbs_cold": mr_bytes / cold / 1e3, "hbm_frac_cold": mr_bytes / cold / 1e3 / PEAK_HBM_GBS,
            "method": f"warm: {reps} back-to-back launches; cold: median(512 MiB write + launch) "
                      f"- median(write alone) over {reps} pairs"}


def measure_config(name, w, api, I, dev, torch, steps: int, warmup: int) -> dict:
    """One workload of the benchmark's configuration set, measured the way the
    headline is: its L-block stack under the one-launch schedule (layers/s),
    every launch of a second pass stamped by its own dispatch (the dominant
    kernel and its roofline), and the two metric components on their own --
    the standalone kNN build (Gram MFMA fraction) and MRConv update (gather
    HBM bandwidth) -- averaged over back-to-back launches with HIP events."""
    import numpy as np
    es = 2 if w.dtype == I.BF16 else 4
    peak = PEAK_TFLOPS[w.dtype]
    x0 = dev(I.make_features(w))
    Wd = dev(I.Stored(np.stack([I.make_weight(w, l).bits for l in range(w.L)]), None, w.dtype))
    bd = dev(I.Stored(np.stack([I.make_bias(w, l).bits for l in range(w.L)]), None, w.dtype))
    s = torch.cuda.current_stream()
    la = api.Lookahead(s, torch.cuda.Stream())
    ws = api.make_stack_workspace(x0, w.H, w.W, w.k, w.pool_r)
    out = torch.empty_like(x0)
    dil = list(w.dilations)

    def step():
        la.stack(x0, w.H, w.W, Wd, bd, dil, w.k, w.pool_r, schedule=api.GL_SCHED_LOOKAHEAD_FUSED,
                 ws=ws, x_out=out)

    def timed(fn, n):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(s)
        for _ in range(n):
            fn()
        e1.record(s)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    for _ in range(warmup):
        step()
    ms = timed(step, steps)
    value = w.L / (ms / 1e3)
    # per-launch durations, stamped by each dispatch on its own stream
    n_rec = steps * w.L + 8
    la.set_profiling(n_rec)
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    times = {key: la.kernel_times_ms(which, n_rec) for key, which in
             (("knn_graph", api.GL_TIME_BUILD), ("mrconv", api.GL_TIME_UPDATE),
              ("graphleap_block", api.GL_TIME_FUSED))}
    la.set_profiling(0)
    la.close()
    knn_flops, knn_bytes, mr_flops, mr_bytes = algorithmic(w, es)
    F, Y = layer_work(w, es)
    pool_io = (w.B * w.N * w.C + w.B * w.M * w.C) * es if w.pool_r > 1 else 0
    kern = {}
    for key, t in times.items():
        if not t:
            continue
        avg = sum(t) / len(t) * 1e-3
        e = {"launches_per_step": len(t) / steps, "avg_us": avg * 1e6, "us_per_step": sum(t) / steps * 1e3}
        if key == "knn_graph":
            e.update(bound="mfma", achieved=knn_flops / avg / 1e12, peak=peak, unit="TFLOP/s")
        elif key == "mrconv":
            e.update(bound="hbm", achieved=mr_bytes / avg / 1e9, peak=PEAK_HBM_GBS, unit="GB/s")
        else:   # one launch = one layer's build and update
            yb = Y - pool_io
            if yb / (PEAK_HBM_GBS * 1e9) >= F / (peak * 1e12):
                e.update(bound="hbm", achieved=yb / avg / 1e9, peak=PEAK_HBM_GBS, unit="GB/s")
            else:
                e.update(bound="mfma", achieved=F / avg / 1e12, peak=peak, unit="TFLOP/s")
        e["frac"] = e["achieved"] / e["peak"]
        kern[key] = e
    dom = max(kern, key=lambda k_: kern[k_]["us_per_step"])
    # the metric's two components, each kernel on its own
    keys = api.pool_keys(x0, w.H, w.W, w.pool_r) if w.pool_r > 1 else None
    idx = torch.empty((w.B, w.N, w.k), dtype=torch.int32, device=x0.device)
    n = max(10, steps // 2)
    t_knn = timed(lambda: api.knn_graph(x0, w.k, dil[-1], keys=keys, out=idx), n) * 1e-3
    mws = api.mrconv_workspace(w.B, w.N, w.C, w.k, w.C, x0.dtype, x0.device)
    t_mr = timed(lambda: api.mrconv(x0, idx, Wd[0], bd[0], keys=keys, out=out, ws=mws), n) * 1e-3
    t_floor = max(F / (peak * 1e12), Y / (PEAK_HBM_GBS * 1e9))
    return {
        "workload": f"{name}: {DESCR[name]}", "dtype": w.dtype, "layers_per_s": value,
        "ms_per_step": ms, "steps": steps, "schedule": "fused",
        "dominant_kernel": {"kernel": dom, **{k_: kern[dom][k_] for k_ in
                                              ("bound", "achieved", "peak", "unit", "frac", "avg_us")}},
        "kernels": kern,
        "gram_mfma": {"kernel": "gl_knn_graph", "d": dil[-1], "avg_us": t_knn * 1e6,
                      "tflops": knn_flops / t_knn / 1e12, "frac": knn_flops / t_knn / 1e12 / peak},
        "gather_hbm": {"kernel": "gl_mrconv", "avg_us": t_mr * 1e6, "gbs": mr_bytes / t_mr / 1e9,
                       "frac": mr_bytes / t_mr / 1e9 / PEAK_HBM_GBS,
                       "effective_gbs": w.B * w.N * w.k * w.C * es / t_mr / 1e9},
        "layer": {"flop": F, "bytes": Y, "roofline_layers_per_s": 1.0 / t_floor,
                  "frac": value * t_floor},
    }


# the benchmark's configuration set besides the headline (one GPU each)
CONFIG_SET = ("single", "vig_b", "pyr_s1", "pyr_s2", "hires")


def full_block(args, w, api, I, dev, torch) -> dict:
    """Time the full ViG block stack (gl_vig_stack) under its three schedules
    and profile its launches."""
    B, N, C = w.B, w.N, w.C
    L = w.L
    x0 = dev(I.make_features(w))
    params = [{n: dev(v) for n, v in I.make_vig_params(w, l).items()} for l in range(L)]
    s_up = torch.cuda.current_stream()
    la = api.Lookahead(s_up, torch.cuda.Stream())
    ws = api.vig_workspace(x0, w.k, w.H, w.W, w.pool_r)
    out = torch.empty_like(x0)
    dil = list(w.dilations)
    steps = max(10, args.steps // 4)

    def run(sc):
        la.vig_stack(x0, params, dil, w.k, schedule=sc, ws=ws, x_out=out, H=w.H, W=w.W,
                     pool_r=w.pool_r)

    def timed(sc, n):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(s_up)
        for _ in range(n):
            run(sc)
        e1.record(s_up)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    res = {}
    for name, sc in (("fused", api.GL_SCHED_LOOKAHEAD_FUSED), ("lookahead", api.GL_SCHED_LOOKAHEAD),
                     ("standard", api.GL_SCHED_STANDARD)):
        for _ in range(max(2, args.warmup // 4)):
            run(sc)
        m = timed(sc, steps)
        res[name] = {"ms_per_step": m, "layers_per_s": L / (m / 1e3)}
    if args.only == "full":
        la.close()
        return {"schedules": res}
    n_rec = steps * L * 5 + 16
    la.set_profiling(n_rec)
    for _ in range(steps):
        run(api.GL_SCHED_LOOKAHEAD_FUSED)
    torch.cuda.synchronize()
    kern = {}
    for key, which in (("linear", api.GL_TIME_LINEAR), ("graphleap_block", api.GL_TIME_FUSED),
                       ("knn_graph", api.GL_TIME_BUILD), ("mrconv", api.GL_TIME_UPDATE)):
        t = la.kernel_times_ms(which, n_rec)
        if t:
            kern[key] = {"launches_per_step": len(t) / steps, "avg_us": sum(t) / len(t) * 1e3,
                         "us_per_step": sum(t) / steps * 1e3}
    la.set_profiling(0)
    la.close()
    # algorithmic flop per layer: Gram + MRConv FC + FC1 + FC2 + FFN (C -> 4C -> C)
    flops = 2.0 * B * N * w.M * C + 2.0 * B * N * C * (2 * C + C + C + 8 * C)
    # the fastest schedule (the same arithmetic and graphs in each); the
    # kernel records above are the fused schedule's
    name = max(res, key=lambda n: res[n]["layers_per_s"])
    best = res[name]
    peak = PEAK_TFLOPS[w.dtype]
    tf = flops / (best["ms_per_step"] / L * 1e-3) / 1e12
    return {"layers_per_s": best["layers_per_s"], "ms_per_step": best["ms_per_step"],
            "schedule": name, "schedules": res, "kernels": kern,
            "flop_per_layer": flops, "tflops": tf, "mfma_frac": tf / peak,
            "entry": "gl_vig_stack"}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="vig_ti")
    ap.add_argument("--schedule", default="fused", choices=["fused", "lookahead", "standard"])
    ap.add_argument("--only", default=None, choices=["stack", "knn", "mrconv", "copy", "full"])
    ap.add_argument("--no-full-block", action="store_true")
    ap.add_argument("--cpu-images", type=int, default=32)
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the other configurations (single, vig_b, pyr_s1, pyr_s2, hires)")
    ap.add_argument("--config-steps", type=int, default=30)
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "the benchmark runs on one GPU only; sharding over GPUs "
                                   "(data-parallel over images) is not implemented",
                          "n_gpus": args.gpus}), flush=True)
        return 2

    import torch

    from paper_2604_21290_amd import api
    from paper_2604_21290_amd import inputs as I

    assert torch.cuda.is_available(), "bench needs a GPU"
    api.lib()
    w = I.WORKLOADS[args.workload]
    es = 2 if w.dtype == I.BF16 else 4
    SCHED = {"fused": api.GL_SCHED_LOOKAHEAD_FUSED, "lookahead": api.GL_SCHED_LOOKAHEAD,
             "standard": api.GL_SCHED_STANDARD}
    sched = SCHED[args.schedule]

    def dev(s):
        import numpy as np
        if s.dtype == I.F32:
            return torch.from_numpy(np.ascontiguousarray(s.bits)).cuda()
        return torch.from_numpy(np.ascontiguousarray(s.bits).view(np.int16)).cuda().view(torch.bfloat16)

    import numpy as np
    x0 = dev(I.make_features(w))
    Wd = dev(I.Stored(np.stack([I.make_weight(w, l).bits for l in range(w.L)]), None, w.dtype))
    bd = dev(I.Stored(np.stack([I.make_bias(w, l).bits for l in range(w.L)]), None, w.dtype))
    s_up = torch.cuda.current_stream()
    la = api.Lookahead(s_up, torch.cuda.Stream())
    ws = api.make_stack_workspace(x0, w.H, w.W, w.k, w.pool_r)
    out = torch.empty_like(x0)
    dil = list(w.dilations)

    if args.only == "copy":
        # plain device copy of a known size, for scaling rocprofv3 FETCH/WRITE counters
        n = 256 << 20
        a = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        b = torch.empty_like(a)
        for _ in range(args.steps):
            b.copy_(a)
        torch.cuda.synchronize()
        log(f"copied {n} bytes x {args.steps}")
        return 0
    if args.only == "full":
        r = full_block(args, w, api, I, dev, torch)
        log("full block", json.dumps(r))
        return 0
    if args.only == "knn":
        keys = api.pool_keys(x0, w.H, w.W, w.pool_r) if w.pool_r > 1 else None
        idx = ws["idx"][0]
        for _ in range(args.steps):
            api.knn_graph(x0, w.k, dil[-1], keys=keys, out=idx)
        torch.cuda.synchronize()
        log(f"knn x {args.steps} (d={dil[-1]})")
        return 0
    if args.only == "mrconv":
        keys = api.pool_keys(x0, w.H, w.W, w.pool_r) if w.pool_r > 1 else None
        idx = api.knn_graph(x0, w.k, dil[0], keys=keys)
        mws = api.mrconv_workspace(w.B, w.N, w.C, w.k, w.C, x0.dtype, x0.device)
        for _ in range(args.steps):
            api.mrconv(x0, idx, Wd[0], bd[0], keys=keys, out=out, ws=mws)
        torch.cuda.synchronize()
        log(f"mrconv x {args.steps}")
        return 0

    def step(sc=None):
        la.stack(x0, w.H, w.W, Wd, bd, dil, w.k, w.pool_r, schedule=sched if sc is None else sc,
                 ws=ws, x_out=out)

    def time_steps(n, sc=None):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(s_up)
        for _ in range(n):
            step(sc)
        e1.record(s_up)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    log(f"workload {args.workload}: warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"timing {args.steps} steps ({args.schedule})")
    t_wall = time.perf_counter()
    ms_per_step = time_steps(args.steps)
    wall = time.perf_counter() - t_wall
    value = w.L / (ms_per_step / 1e3)
    log(f"{ms_per_step:.4f} ms/step, {value:.1f} layers/s (wall {wall:.3f} s)")

    # the other schedules, same kernels, for context
    schedules = {args.schedule: {"ms_per_step": ms_per_step, "layers_per_s": value}}
    if args.only != "stack":
        for name, sc in SCHED.items():
            if name == args.schedule:
                continue
            for _ in range(max(2, args.warmup // 4)):
                step(sc)
            m = time_steps(max(10, args.steps // 4), sc)
            schedules[name] = {"ms_per_step": m, "layers_per_s": w.L / (m / 1e3)}
        g = graph_replay(args, w, api, torch, x0, Wd, bd, dil, ws, out)
        if g is not None:
            schedules["fused_hip_graph"] = g
        log("schedules", json.dumps(schedules))
        # build/update overlap: the serial schedule against the two overlapped ones
        t_ser = schedules["standard"]["ms_per_step"]
        overlap = {"serial_over_lookahead": t_ser / schedules["lookahead"]["ms_per_step"],
                   "serial_over_fused": t_ser / schedules["fused"]["ms_per_step"]}
        per_step = step_percentiles(torch, step, s_up, args.steps)
        log("per-stack times", json.dumps(per_step))

    # per-kernel durations: the same steps again, every launch stamped with a
    # start and an end HIP event by its own dispatch, on its own stream
    if args.only == "stack":
        return 0
    n_rec = args.steps * w.L + 8
    la.set_profiling(n_rec)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    tb = la.kernel_times_ms(api.GL_TIME_BUILD, n_rec)
    tu = la.kernel_times_ms(api.GL_TIME_UPDATE, n_rec)
    tf = la.kernel_times_ms(api.GL_TIME_FUSED, n_rec)
    la.set_profiling(0)
    knn_flops, knn_bytes, mr_flops, mr_bytes = algorithmic(w, es)
    peak = PEAK_TFLOPS[w.dtype]
    kernels = {}
    if tb:
        t = sum(tb) / len(tb) * 1e-3
        kernels["knn_graph"] = {
            "launches_per_step": len(tb) / args.steps, "avg_us": t * 1e6,
            "gram_tflops": knn_flops / t / 1e12, "gram_mfma_frac": knn_flops / t / 1e12 / peak,
            "candidates_per_s": w.B * w.N * w.M / t}
    if tu:
        t = sum(tu) / len(tu) * 1e-3
        kernels["mrconv"] = {
            "launches_per_step": len(tu) / args.steps, "avg_us": t * 1e6,
            "fc_tflops": mr_flops / t / 1e12, "fc_mfma_frac": mr_flops / t / 1e12 / peak,
            "hbm_gbs": mr_bytes / t / 1e9, "hbm_frac": mr_bytes / t / 1e9 / PEAK_HBM_GBS,
            "gather_effective_gbs": (w.B * w.N * w.k * w.C * es) / t / 1e9}
    # one-launch block = one layer: the layer's algorithmic bytes (X read by the
    # build and again by the update, the graph written and read, W, X^(l+1)
    # written); the block's own floor (X read once by both roles) is reported
    # beside it
    fb_flops, fb_bytes = layer_work(w, es)
    fb_bytes -= (w.B * w.N * w.C + w.B * w.M * w.C) * es if w.pool_r > 1 else 0
    fb_floor = mr_bytes + w.B * w.N * w.k * 4
    if tf:
        t = sum(tf) / len(tf) * 1e-3
        kernels["graphleap_block"] = {
            "launches_per_step": len(tf) / args.steps, "avg_us": t * 1e6,
            "tflops": fb_flops / t / 1e12, "mfma_frac": fb_flops / t / 1e12 / peak,
            "hbm_gbs": fb_bytes / t / 1e9, "hbm_frac": fb_bytes / t / 1e9 / PEAK_HBM_GBS,
            "block_floor_bytes": fb_floor, "block_floor_hbm_frac": fb_floor / t / 1e9 / PEAK_HBM_GBS}
    totals = {"knn_graph": sum(tb), "mrconv": sum(tu), "graphleap_block": sum(tf)}
    dom = max(totals, key=totals.get)
    if dom == "knn_graph":
        t = sum(tb) / len(tb) * 1e-3
        roof = {"kernel": "knn_graph", "bound": "mfma", "achieved": knn_flops / t / 1e12,
                "peak": peak, "unit": "TFLOP/s", "frac": knn_flops / t / 1e12 / peak,
                "traffic": load_traffic("knn_graph", args.workload),
                "per_launch": f"Gram 2*B*N*M*C = {knn_flops:.4g} flop"}
    elif dom == "mrconv":
        t = sum(tu) / len(tu) * 1e-3
        roof = {"kernel": "mrconv", "bound": "hbm", "achieved": mr_bytes / t / 1e9,
                "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": mr_bytes / t / 1e9 / PEAK_HBM_GBS,
                "traffic": load_traffic("mrconv", args.workload),
                "per_launch": f"{mr_bytes:.4g} bytes"}
    else:
        t = sum(tf) / len(tf) * 1e-3
        if fb_bytes / (PEAK_HBM_GBS * 1e9) >= fb_flops / (peak * 1e12):
            roof = {"kernel": "graphleap_block", "bound": "hbm", "achieved": fb_bytes / t / 1e9,
                    "peak": PEAK_HBM_GBS, "unit": "GB/s",
                    "frac": fb_bytes / t / 1e9 / PEAK_HBM_GBS,
                    "traffic": load_traffic("graphleap_block", args.workload),
                    "per_launch": f"{fb_bytes:.4g} bytes = one layer's algorithmic bytes (X read by "
                                  f"the build and by the update, graph written and read, W, output); "
                                  f"flop floor {fb_flops:.4g}",
                    "block_floor": {"bytes": fb_floor, "frac": fb_floor / t / 1e9 / PEAK_HBM_GBS,
                                    "note": "X read once by both roles of the one launch"}}
        else:
            roof = {"kernel": "graphleap_block", "bound": "mfma", "achieved": fb_flops / t / 1e12,
                    "peak": peak, "unit": "TFLOP/s", "frac": fb_flops / t / 1e12 / peak,
                    "traffic": load_traffic("graphleap_block", args.workload),
                    "per_launch": f"{fb_flops:.4g} flop (byte floor {fb_bytes:.4g})"}
    log("kernels", json.dumps(kernels))
    if "mrconv" in kernels or "graphleap_block" in kernels:
        kernels.setdefault("mrconv", {})["cold_cache"] = cold_gather(
            w, api, torch, x0, ws["idx"][0], Wd[0], bd[0], out, mr_bytes)
        log("mrconv warm/cold", json.dumps(kernels["mrconv"]["cold_cache"]))
    # the whole layer against its roofline: F = Gram + FC flop, Y = the block's byte floor
    t_floor = max(fb_flops / (peak * 1e12), fb_bytes / (PEAK_HBM_GBS * 1e9))
    layer_roofline = {"layers_per_s": 1.0 / t_floor, "frac": value * t_floor,
                      "flop_per_layer": fb_flops, "bytes_per_layer": layer_work(w, es)[1]}
    st = stage_transition(w, api, torch, x0, es)
    if st is not None:
        kernels["stage_transition"] = st
        log("stage transition", json.dumps(st))
    hu = heads_update(args, w, api, torch, x0, ws["idx"][0], Wd[0])
    if hu is not None:
        kernels["mrconv_heads"] = hu
        log("multi-head update", json.dumps(hu))

    full = None
    if not args.no_full_block:
        log("full ViG block stack")
        full = full_block(args, w, api, I, dev, torch)
        log("full block", json.dumps(full))

    configs = None
    if not args.no_configs and args.workload == "vig_ti":
        configs = {}
        for name in CONFIG_SET:
            log(f"config {name}")
            configs[name] = measure_config(name, I.WORKLOADS[name], api, I, dev, torch,
                                           steps=args.config_steps, warmup=max(2, args.config_steps // 5))
            c = configs[name]
            log(f"  {c['layers_per_s']:.0f} layers/s; dominant {c['dominant_kernel']['kernel']} "
                f"{100 * c['dominant_kernel']['frac']:.2f}% of {c['dominant_kernel']['bound']}; "
                f"Gram {100 * c['gram_mfma']['frac']:.2f}% MFMA; gather {c['gather_hbm']['gbs']:.0f} GB/s")

    cpu = None
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle)")
        cpu = cpu_baseline(w, args.cpu_images, args.cpu_seconds)
        log("cpu", json.dumps(cpu))
        if full is not None:
            full["cpu_oracle"] = cpu_full_block(w, 2, min(w.L, 4))
            log("cpu full block", json.dumps(full["cpu_oracle"]))

    line = {
        "metric": METRIC, "value": value, "unit": "layers/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": f"{args.workload}: {DESCR[args.workload]}", "B": w.B, "N": w.N,
                   "M": w.M, "C": w.C, "k": w.k, "blocks": w.L, "dilations": dil,
                   "schedule": args.schedule},
        "roofline": roof, "cpu_baseline": cpu, "kernels": kernels, "schedules": schedules,
        "full_block": full, "per_stack": per_step, "overlap": overlap, "layer_roofline": layer_roofline,
        "image_layers_per_s": value * w.B, "configs": configs, "source_sha": kernel_source_sha(),
    }
    print(json.dumps(line), flush=True)
    la.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
