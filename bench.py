#!/usr/bin/env python
"""Benchmark of the MonarchAttention forward pass on one MI355X.

One step = one monarch_attn_fwd call: the whole forward pass (every R and L
half-step, the Monarch product and the store of O) over one batch of
synthetic Q, K, V already resident in HBM.  The headline workload is the
long-sequence speed point (B=1, H=16, N=16384 = 128 x 128, d=64, bf16, T=2);
the medium point (N=4096 = 64 x 64, T=1 and T=3) and ViT-B/16 (384 heads, N=196 = 14 x 14,
T=2, the one-workgroup-per-head kernel; and N=197 with the class token,
post-padded to 15 x 14) and RoBERTa-base-shaped attention (192 heads, N=1024
= 32 x 32, T=2, the grouped kernel) are reported alongside in "also".

Timed regions (HIP events on the stream the library launches on):
  0. (untimed) W warm-up steps, repeated in rounds of W until 0.25 s of
     calls have run, so that the GPU has left its idle clocks.
  1. K steps back to back -> ms_per_step and value = B*H*N / time.
  2. K more steps with the library's per-launch events enabled -> the average
     duration of each kernel.  A pair of events adds a roughly fixed time to
     every launch it brackets (about 2.5 us here), so each duration has the
     per-launch excess of the event-read step over the step of region 1 taken
     off (launch_overhead_us; the raw reading is kept as event_us).
Inputs rotate over several copies (>= 512 MB in total) so that the 256 MB
last-level cache cannot serve them from one step to the next.

`roofline` is that of the whole call: the compulsory bytes 4 N d s per head
(Q, K, V read once, O written once) over the call time against 8 TB/s, or
the method's flops against the MFMA peak when those bound it.  `traffic` is
the HBM bytes one call moves by the committed rocprofv3 counters (null once
a kernel's sources changed since they were taken).  The dominant kernel
(largest share of the step) is named beside it with its fraction on the
bytes of the paper's state organisation (design IO), a secondary figure.

The last line of stdout is one compact JSON record (< 4 KB): the headline,
its roofline, the CPU baseline and a short line per extra workload.  The full
record (per-kernel times, per-call distributions, hot and graph-replayed
times, the sweep, the gradient, padded batches and quality) goes to the file
named by --details.

Each workload also reports the p10 / median / p90 of single calls (each
between its own events), a "hot" time on one input set, and the time per call
when the rotating calls are captured into a HIP graph and replayed (no host
launch cost; graph_ms_per_call).  measured_peaks
holds a 1 GiB device copy and 8192^3 GEMMs (bf16, fp32) timed on this GPU;
every roofline record adds its fraction of that measured peak beside the
fraction of the published one.

sweep: the long-sequence points N = 256, 1024, 4096, 16384 (sqrt(N) x
sqrt(N), d = 64 and 128, T = 2, 16 heads), with the call roofline and the
dominant kernel of each.  With --sdpa, at d = 64 and the paper's quoted N it
also times torch's fused scaled_dot_product_attention on the same shape, as
context beside the paper's own speed-ups over FlashAttention-2 on its
hardware (off by default: a comparison system, not part of the method).

cpu_baseline: the fp64 C oracle, as it stands, on this host's cores, on the
same workload (repeated whole forward passes, about 10-15 s in total).

backward: monarch_attn_bwd (the gradient: forward recompute keeping every
step's states, then the reverse sweep) timed the same way on the 4K speed
point and ViT-B/16 with its class token, with its per-kernel durations and
the roofline of its dominant gradient kernel.  In the details file only.

varlen: monarch_attn_fwd_varlen and monarch_attn_bwd_varlen on a padded
batch (RoBERTa-base shape at N = 384, b = 48, T = 1; lengths iid uniform on
64..384), each beside the plain call on the same tensors.

quality: the error of O against exact softmax attention and the gap of the
variational objective to its exact-softmax maximum, for T = 1, 2, 3, on the
structured workloads (ViT- and RoBERTa-shaped, and 16K tokens with
RoBERTa-like decaying scores; the speed points' iid Q, K have no structure
to approximate).  GPU only, outside the timed regions.

Only one GPU is supported: --gpus N with N > 1 exits with a message.
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MonarchAttention fwd heads*tokens/sec + % MFMA/HBM roofline at N=4K,16K"
UNIT = "heads*tokens/s"
HBM_PEAK_GBS = 8000.0            # MI355X HBM3E, GB/s
MFMA_PEAK_TFLOPS = {"bf16": 2516.6, "f16": 2516.6, "f32": 157.3}
ROTATE_BYTES = 512 << 20


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def launch_plan(w):
    """The kernels of one call in launch order, with the algorithmic bytes and
    flops each moves and computes (all heads).

    Bytes count each state or tensor element once per kernel that reads or
    writes it: R half-step reads alpha_R (Q at t=1) and K, writes alpha_L and
    c_L (reads c_R after t=1); the last one also reads V and writes Y.  The L
    half-step reads Q, alpha_L, c_L and writes alpha_R, c_R.  The apply reads
    Q, alpha_L, Y, c_L and writes O.  Flops are 2 per multiply-add of the
    products (beta and alpha contractions, Y and O).  Tensors have N rows per
    head; states and flops cover the Np = m * b rows of the padded sequence
    (Np = N unless N is not a multiple of b).
    """
    s = 2 if w.dtype in ("bf16", "f16") else 4
    BH, N, d, m, b = w.B * w.H, w.N, w.d, w.m, w.b
    Np = m * b
    nd, sd = N * d * s, Np * d * s   # one tensor, one state
    plan = []
    for t in range(1, w.T + 1):
        first, last = t == 1, t == w.T
        # R: alpha_R (Q at t=1), K in; alpha_L, c_L out; c_R in after t=1; V in, Y out when last
        rb = (nd if first else sd) + nd + sd + 4 * Np + (0 if first else 4 * Np)
        rf = 2 * 2 * Np * b * d
        if last:
            rb += nd + sd
            rf += 2 * Np * b * d
        plan.append(("r_half_step_final" if last else "r_half_step", BH * rb, BH * rf))
        if last:  # Q, alpha_L, Y, c_L in; O out
            plan.append(("monarch_apply", BH * (2 * nd + 2 * sd + 4 * Np), BH * 2 * 2 * Np * m * d))
        else:     # Q, alpha_L, c_L in; alpha_R, c_R out
            plan.append(("l_half_step", BH * (nd + 2 * sd + 8 * Np), BH * 2 * 2 * Np * m * d))
    return plan


def plan_for(w, kinds):
    """Launch plan matching the kernels one call actually ran."""
    if kinds in (["monarch_fused_head"], ["monarch_fused_group"]):
        # one launch for the whole pass: its algorithmic traffic is the compulsory
        # Q, K, V in and O out (the states stay in LDS)
        compulsory, flops = call_work(w)
        return [(kinds[0], compulsory, flops)]
    plan = launch_plan(w)
    assert kinds == [p[0] for p in plan], (kinds, plan)
    return plan


WARM_S = 0.25  # seconds of untimed calls before a timed region (at least W calls)


def warm_up(torch, step, warmup):
    """W untimed calls, repeated in rounds of W until they have kept the GPU
    busy for WARM_S seconds: after an idle spell (input generation, the
    previous workload's host work) the GPU takes several milliseconds of work
    to reach its steady clocks, and the timed region should see those.
    W = 0 runs nothing."""
    if warmup <= 0:
        return
    t0, i = time.perf_counter(), 0
    while True:
        for _ in range(warmup):
            step(i)
            i += 1
        torch.cuda.synchronize()
        if time.perf_counter() - t0 >= WARM_S:
            return


def launch_overhead_ms(event_ms, step_ms):
    """Per-launch cost of the per-launch events: each launch's pair of events
    adds a roughly fixed time (dispatch after the first event, completion
    before the second) to the duration it reads.  Estimated as the excess of
    the event-read durations of one step over the un-instrumented step time,
    shared equally over the step's launches (0 if there is none); subtracting
    it leaves each kernel the time it took in the timed region, gaps between
    launches included."""
    return max(0.0, (sum(event_ms) - step_ms) / len(event_ms)) if event_ms else 0.0


def call_work(w):
    """Compulsory bytes (Q, K, V in, O out: N rows) and flops of the method
    (on the Np = m * b rows it runs over) of one call."""
    s = 2 if w.dtype in ("bf16", "f16") else 4
    BH, Np = w.B * w.H, w.m * w.b
    compulsory = BH * 4 * w.N * w.d * s
    macs = w.T * (2 * Np * w.b * w.d + 2 * Np * w.m * w.d) + Np * w.b * w.d
    return compulsory, 2 * BH * macs


def measure(ma, torch, w, steps, warmup):
    import synth_inputs as si

    t0 = time.time()
    q, k, v, meta = si.make_qkv(w)
    log(f"[bench] {w.name}: inputs generated in {time.time() - t0:.1f}s")
    td = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}[w.dtype]
    base = [torch.from_numpy(x).to(td).cuda() for x in (q, k, v)]
    del q, k, v
    set_bytes = 4 * base[0].numel() * base[0].element_size()
    nsets = max(1, min(8, math.ceil(ROTATE_BYTES / set_bytes)))
    sets = [(base[0].clone(), base[1].clone(), base[2].clone(), torch.empty_like(base[0])) for _ in range(nsets)]
    del base

    def step(i):
        qq, kk, vv, oo = sets[i % nsets]
        ma.monarch_attn_fwd(qq, kk, vv, oo, w.m, w.b, w.T)

    warm_up(torch, step, warmup)
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for i in range(steps):
        step(i)
    end.record()
    end.synchronize()
    ms = start.elapsed_time(end) / steps
    log(f"[bench] {w.name}: {ms * 1e3:.1f} us per step over {steps} steps ({nsets} rotating input sets)")
    extra = {"per_call_us": per_call_distribution(torch, step, steps), "hot_ms_per_step": hot_time(torch, step, steps),
             "graph_ms_per_call": graph_time(torch, step, steps, nsets)}

    # per-launch kernel durations
    plan, sums = None, None
    ma.monarch_attn_timing_enable(True)
    try:
        for i in range(steps):
            step(i)
            recs = ma.monarch_attn_timing_read()
            if plan is None:
                plan = plan_for(w, [kind for kind, _ in recs])
                sums = [0.0] * len(plan)
            assert [kind for kind, _ in recs] == [p[0] for p in plan], (recs, plan)
            for j, (kind, t) in enumerate(recs):
                sums[j] += t
    finally:
        ma.monarch_attn_timing_enable(False)
    kernels = []
    over = launch_overhead_ms([t / steps for t in sums], ms)
    extra["launch_overhead_us"] = round(over * 1e3, 3)
    for (name, nbytes, nflops), tot in zip(plan, sums):
        avg_ms = tot / steps - over
        kernels.append({
            "kernel": name,
            "avg_us": round(avg_ms * 1e3, 3),
            "event_us": round(tot / steps * 1e3, 3),
            "alg_bytes": nbytes,
            "alg_flops": nflops,
            "GB_s": round(nbytes / (avg_ms * 1e-3) / 1e9, 1),
            "TFLOP_s": round(nflops / (avg_ms * 1e-3) / 1e12, 2),
        })
    torch.cuda.synchronize()
    del sets
    torch.cuda.empty_cache()
    return ms, kernels, meta, nsets, extra


def per_call_distribution(torch, step, steps):
    """p10 / median / p90 of single calls, each between its own pair of events
    (rotating inputs as in the main region)."""
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for i, (a, b) in enumerate(evs):
        a.record()
        step(i)
        b.record()
    torch.cuda.synchronize()
    t = sorted(a.elapsed_time(b) * 1e3 for a, b in evs)

    def q(f):
        return round(t[min(len(t) - 1, int(f * (len(t) - 1) + 0.5))], 3)

    return {"p10": q(0.1), "p50": q(0.5), "p90": q(0.9)}


def hot_time(torch, step, steps):
    """ms per call with the same input set every call (caches warm), labelled hot."""
    step(0)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(steps):
        step(0)
    b.record()
    b.synchronize()
    return round(a.elapsed_time(b) / steps, 6)


def graph_time(torch, step, steps, nsets):
    """ms per call when one call per input set is captured into a HIP graph
    and the graph is replayed: the calls' GPU time without the host's launch
    and binding cost.  The capture stream's workspace is sized by an eager
    call on it first (a call under capture does not allocate)."""
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        for i in range(nsets):
            step(i)
    s.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        for i in range(nsets):
            step(i)
    reps = max(1, -(-steps // nsets))
    g.replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        g.replay()
    b.record()
    b.synchronize()
    ms = a.elapsed_time(b) / (reps * nsets)
    del g
    return round(ms, 6)


def measured_peaks(torch):
    """Peaks measured on this GPU, beside the published ones: a 1 GiB device copy
    (read + write bytes / time) and dense 8192^3 GEMMs through torch (hipBLASLt)
    in bf16 and fp32.  Context for the roofline fractions, not a substitute."""
    out = {}
    n = (1 << 30) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(10):
        dst.copy_(src)
    b.record()
    b.synchronize()
    out["copy_GB_s"] = round(2 * n * 4 * 10 / (a.elapsed_time(b) * 1e-3) / 1e9, 1)
    del src, dst
    for name, dt in (("gemm_bf16_TFLOP_s", torch.bfloat16), ("gemm_f32_TFLOP_s", torch.float32)):
        x = torch.randn(8192, 8192, device="cuda").to(dt)
        y = torch.randn(8192, 8192, device="cuda").to(dt)
        for _ in range(2):
            torch.matmul(x, y)
        a.record()
        for _ in range(5):
            torch.matmul(x, y)
        b.record()
        b.synchronize()
        out[name] = round(2 * 8192 ** 3 * 5 / (a.elapsed_time(b) * 1e-3) / 1e12, 1)
        del x, y
    torch.cuda.empty_cache()
    return out


def with_measured(roof, peaks):
    """Add the fraction of the measured peak to a roofline record."""
    if peaks:
        key = "copy_GB_s" if roof["unit"] == "GB/s" else (
            "gemm_f32_TFLOP_s" if roof["peak"] == MFMA_PEAK_TFLOPS["f32"] else "gemm_bf16_TFLOP_s")
        roof["measured_peak"] = peaks[key]
        roof["frac_of_measured"] = round(roof["achieved"] / peaks[key], 4)
    return roof


# The paper's speed-ups of MonarchAttention over FlashAttention-2 (its own
# hardware and Triton kernels), quoted as context beside the same ratio on this
# GPU against torch's fused attention.
PAPER_SPEEDUP_VS_FA2 = {256: 1.4, 4096: 4.5, 16384: 8.2}


def sdpa_context(ma, torch, w, steps, warmup, monarch_ms):
    """Time torch.nn.functional.scaled_dot_product_attention (flash or
    memory-efficient backend only, never the math path) on the workload's
    shape with rotating inputs, and the ratio to the Monarch call."""
    import torch.nn.functional as F
    from torch.nn.attention import SDPBackend, sdpa_kernel

    shape = (w.B, w.H, w.N, w.d)
    per_set = 4 * w.B * w.H * w.N * w.d * 2
    nsets = max(1, min(8, math.ceil(ROTATE_BYTES / per_set)))
    sets = [[torch.randn(shape, device="cuda", dtype=torch.bfloat16) for _ in range(3)] for _ in range(nsets)]
    res = {"N": w.N, "paper_speedup_vs_fa2": PAPER_SPEEDUP_VS_FA2.get(w.N)}
    for backend in (SDPBackend.FLASH_ATTENTION, SDPBackend.EFFICIENT_ATTENTION):
        try:
            with sdpa_kernel(backend):
                warm_up(torch, lambda i: F.scaled_dot_product_attention(*sets[i % nsets]), warmup)
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record()
                for i in range(steps):
                    F.scaled_dot_product_attention(*sets[i % nsets])
                b.record()
                b.synchronize()
            ms = a.elapsed_time(b) / steps
            res.update({"sdpa_backend": backend.name, "sdpa_ms": round(ms, 6), "monarch_ms": round(monarch_ms, 6),
                        "speedup": round(ms / monarch_ms, 3)})
            break
        except RuntimeError as e:
            res[f"{backend.name}_unavailable"] = str(e).splitlines()[0][:160]
    del sets
    torch.cuda.empty_cache()
    return res


def bwd_kernel_work(w, kind, t):
    """Algorithmic bytes and flops of one gradient launch (all heads) at step t.

    l_bwd (per class j, m x m x d products: scores, dL, dY or L d alpha_R',
    dQ, d alpha_L) reads Q, alpha_L and Y + dO (t = T) or d alpha_R' + d c_R'
    (fp32), and c_L; writes dQ (fp32; read and written when t < T),
    d alpha_L, d c_L and dY (t = T).  r_bwd (per block k, b x b x d products:
    scores, dR (+ dY V^T at t = T), d alpha_R, two for dK, dV at t = T) reads
    K, alpha_R (Q at t = 1), c_R, d alpha_L, d c_L, and V + dY at t = T;
    writes d alpha_R + d c_R (t > 1), dK (fp32, read too unless t = T), and
    at t = 1 reads dQ and writes dq, dk in the element type, at t = T dv.
    Only the d real columns count; the states are stored 64 wide."""
    s = 2 if w.dtype in ("bf16", "f16") else 4
    BH, Np, d, m, b, T = w.B * w.H, w.m * w.b, w.d, w.m, w.b, w.T
    rows = BH * Np
    if kind == "l_bwd":
        macs = 5 * rows * m * d
        if t == T:
            nbytes = rows * d * (4 * s + 12) + rows * 8
        else:
            nbytes = rows * d * (2 * s + 16) + rows * 12
    else:
        macs = (7 if t == T else 5) * rows * b * d
        nbytes = rows * (2 * d * s + d * 4 + 4)        # K, alpha_R (Q at t = 1), d alpha_L, d c_L
        if t > 1:
            nbytes += rows * (4 + d * 4 + 4)           # c_R in; d alpha_R, d c_R out
        if t == T:
            nbytes += rows * d * (s + 4 + s)           # V, dY in; dv out
        if t == 1:
            nbytes += rows * d * (4 + s)               # dQ in, dq out
            nbytes += rows * d * ((4 if T > 1 else 0) + s)   # dK in (when accumulated), dk out
        else:
            nbytes += rows * d * 4 * (1 if t == T else 2)    # dK accumulator written (and read when t < T)
    return nbytes, 2 * macs


def measure_backward(ma, torch, w, steps, warmup):
    """Time monarch_attn_bwd: K calls back to back, then K with per-launch events."""
    import synth_inputs as si

    q, k, v, _ = si.make_qkv(w)
    dout = si.random_cotangent((w.B, w.H, w.N, w.d), w.dtype, seed=1)
    td = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}[w.dtype]
    base = [torch.from_numpy(x).to(td).cuda() for x in (q, k, v, dout)]
    del q, k, v, dout
    set_bytes = 7 * base[0].numel() * base[0].element_size()
    nsets = max(1, min(8, math.ceil(ROTATE_BYTES / set_bytes)))
    sets = [[x.clone() for x in base] + [torch.empty_like(base[0]) for _ in range(3)] for _ in range(nsets)]
    del base

    def step(i):
        ma.monarch_attn_bwd(*sets[i % nsets], w.m, w.b, w.T)

    warm_up(torch, step, warmup)
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for i in range(steps):
        step(i)
    end.record()
    end.synchronize()
    ms = start.elapsed_time(end) / steps
    log(f"[bench] backward {w.name} T{w.T}: {ms * 1e3:.1f} us per call over {steps} calls")

    kinds, sums = None, None
    ma.monarch_attn_timing_enable(True)
    try:
        for i in range(steps):
            step(i)
            recs = ma.monarch_attn_timing_read()
            if kinds is None:
                kinds = [kind for kind, _ in recs]
                sums = [0.0] * len(kinds)
            assert [kind for kind, _ in recs] == kinds, (recs, kinds)
            for j, (_, t) in enumerate(recs):
                sums[j] += t
    finally:
        ma.monarch_attn_timing_enable(False)
    torch.cuda.synchronize()
    del sets
    torch.cuda.empty_cache()

    # the recompute's launches follow the forward's plan (without the apply);
    # the sweep runs t = T .. 1 as (l_bwd, r_bwd) pairs
    fwd_plan = [p for p in launch_plan(w) if p[0] != "monarch_apply"]
    nrec = len(fwd_plan)
    assert kinds[:nrec] == [p[0] for p in fwd_plan], (kinds, fwd_plan)
    kernels = []
    over = launch_overhead_ms([t / steps for t in sums], ms)
    for j, kind in enumerate(kinds):
        avg_ms = sums[j] / steps - over
        if j < nrec:
            nbytes, nflops = fwd_plan[j][1], fwd_plan[j][2]
            step_t = None
        else:
            step_t = w.T - (j - nrec) // 2
            nbytes, nflops = bwd_kernel_work(w, kind, step_t)
        kernels.append({"kernel": kind, "step": step_t, "avg_us": round(avg_ms * 1e3, 3),
                        "event_us": round(sums[j] / steps * 1e3, 3), "alg_bytes": nbytes,
                        "alg_flops": nflops, "GB_s": round(nbytes / (avg_ms * 1e-3) / 1e9, 1),
                        "TFLOP_s": round(nflops / (avg_ms * 1e-3) / 1e12, 2)})
    sweep = kernels[nrec:]
    dom = max(sweep, key=lambda x: x["avg_us"])
    # the sweep's products are fp32 MFMA whatever the element type
    roof = roofline_of(dom, "f32")
    roof["traffic"] = measured_traffic(f"{dom['kernel']}[t={dom['step']}]", w.name)
    return {"config": w.describe(), "value": round(w.B * w.H * w.N / (ms * 1e-3), 1), "unit": UNIT,
            "ms_per_call": round(ms, 6), "recompute_us": round(sum(x["avg_us"] for x in kernels[:nrec]), 3),
            "sweep_us": round(sum(x["avg_us"] for x in sweep), 3), "roofline": roof, "kernels": kernels,
            "launch_overhead_us": round(over * 1e3, 3), "rotating_input_sets": nsets}


QUALITY_WORKLOADS = ("vit_b16_n196", "roberta_n1024", "lm_n16384")


def time_calls(torch, step, steps, warmup):
    """ms per call of `step(i)` over `steps` calls back to back, after the warm-up."""
    warm_up(torch, step, warmup)
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for i in range(steps):
        step(i)
    end.record()
    end.synchronize()
    return start.elapsed_time(end) / steps


def kernel_times(ma, step, steps):
    """Average duration (us) of each launch of `step`, from the library's
    per-launch events, in launch order."""
    sums, names = None, None
    ma.monarch_attn_timing_enable(True)
    try:
        for i in range(steps):
            step(i)
            recs = ma.monarch_attn_timing_read()
            if sums is None:
                names, sums = [kind for kind, _ in recs], [0.0] * len(recs)
            for j, (_, t) in enumerate(recs):
                sums[j] += t
    finally:
        ma.monarch_attn_timing_enable(False)
    return [[name, round(t / steps * 1e3, 3)] for name, t in zip(names, sums)]


def measure_varlen(ma, torch, w, steps, warmup, low=64):
    """monarch_attn_fwd_varlen over a padded batch of w's shape with lengths
    iid uniform on low..N (seed 0), and the plain call on the same tensors."""
    import synth_inputs as si

    q, k, v, meta = si.make_qkv(w)
    lens_np = si.sequence_lengths(w.B, w.N, seed=0, low=min(low, w.N))
    td = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}[w.dtype]
    base = [torch.from_numpy(x).to(td).cuda() for x in (q, k, v)]
    del q, k, v
    lens = torch.from_numpy(lens_np).cuda()
    set_bytes = 4 * base[0].numel() * base[0].element_size()
    nsets = max(1, min(8, math.ceil(ROTATE_BYTES / set_bytes)))
    sets = [(base[0].clone(), base[1].clone(), base[2].clone(), torch.empty_like(base[0])) for _ in range(nsets)]
    del base

    def step_varlen(i):
        qq, kk, vv, oo = sets[i % nsets]
        ma.monarch_attn_fwd_varlen(qq, kk, vv, oo, lens, w.m, w.b, w.T)

    def step_plain(i):
        qq, kk, vv, oo = sets[i % nsets]
        ma.monarch_attn_fwd(qq, kk, vv, oo, w.m, w.b, w.T)

    ms = time_calls(torch, step_varlen, steps, warmup)
    ms_plain = time_calls(torch, step_plain, steps, warmup)
    kern, kern_plain = kernel_times(ma, step_varlen, steps), kernel_times(ma, step_plain, steps)

    # the gradient of the same padded batch, beside the plain gradient
    dout = torch.from_numpy(si.random_cotangent((w.B, w.H, w.N, w.d), w.dtype, seed=0)).to(td).cuda()
    grads = [torch.empty_like(sets[0][0]) for _ in range(3)]

    def bwd_varlen(i):
        qq, kk, vv, _ = sets[i % nsets]
        ma.monarch_attn_bwd_varlen(qq, kk, vv, dout, *grads, lens, w.m, w.b, w.T)

    def bwd_plain(i):
        qq, kk, vv, _ = sets[i % nsets]
        ma.monarch_attn_bwd(qq, kk, vv, dout, *grads, w.m, w.b, w.T)

    ms_bwd = time_calls(torch, bwd_varlen, steps, warmup)
    ms_bwd_plain = time_calls(torch, bwd_plain, steps, warmup)
    del sets, dout, grads
    torch.cuda.empty_cache()
    real = int(lens_np.sum())
    cfg = w.describe()
    cfg.update({"lengths": f"iid uniform on {min(low, w.N)}..{w.N}, seed 0", "real_rows": real,
                "padded_rows": w.B * w.N, "rotating_input_sets": nsets})
    log(f"[bench] varlen {w.name}: {ms * 1e3:.1f} us per call (plain call {ms_plain * 1e3:.1f} us), "
        f"gradient {ms_bwd * 1e3:.1f} us (plain {ms_bwd_plain * 1e3:.1f} us), {real} of {w.B * w.N} rows real")
    return {"config": cfg, "value": round(w.B * w.H * w.N / (ms * 1e-3), 1), "unit": UNIT,
            "ms_per_call": round(ms, 6), "plain_ms_per_call": round(ms_plain, 6),
            "real_heads_tokens_per_s": round(w.H * real / (ms * 1e-3), 1),
            "kernels_us": kern, "plain_kernels_us": kern_plain,
            "gradient_ms_per_call": round(ms_bwd, 6), "plain_gradient_ms_per_call": round(ms_bwd_plain, 6)}


def quality(ma, torch, w, steps_list=(1, 2, 3)):
    """Approximation quality on the workload's first input set, all on the GPU:
    the relative Frobenius error of O against exact softmax attention
    (monarch_attn_exact_fwd), and the objective gap per query row,
    (sum of exact row logsumexps - f(M^(T))) / N in nats, for several T.
    The exact kernel is this library's reference, not a tuned attention
    kernel; its time is context only."""
    import synth_inputs as si

    q, k, v, _ = si.make_qkv(w)
    td = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}[w.dtype]
    t = [torch.from_numpy(x).to(td).cuda() for x in (q, k, v)]
    del q, k, v
    exact = torch.empty_like(t[0])
    lse = torch.empty(t[0].shape[:3], dtype=torch.float32, device="cuda")
    ma.monarch_attn_exact_fwd(t[0], t[1], t[2], exact, lse)
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    ma.monarch_attn_exact_fwd(t[0], t[1], t[2], exact, lse)
    end.record()
    end.synchronize()
    ex = exact.double()
    bound = lse.double().sum(dim=2)   # [B, H]
    rows = []
    for T in steps_list:
        out = torch.empty_like(t[0])
        obj = torch.empty((w.B, w.H, T), dtype=torch.float32, device="cuda")
        ma.monarch_attn_fwd_objective(t[0], t[1], t[2], out, obj, w.m, w.b, T)
        torch.cuda.synchronize()
        err = float(torch.linalg.vector_norm(out.double() - ex) / torch.linalg.vector_norm(ex))
        gap = ((bound - obj[..., -1].double()) / w.N).mean().item()
        rows.append({"T": T, "rel_frob_vs_exact": round(err, 5), "objective_gap_per_row": round(gap, 5),
                     "objective_per_step": [round(x, 2) for x in obj[0, 0].tolist()]})
    torch.cuda.synchronize()
    return {"workload": w.name, "exact_us": round(start.elapsed_time(end) * 1e3, 1),
            "exact_objective_head0": round(float(bound[0, 0]), 2), "monarch": rows}


# Sources whose text fixes each kernel's memory traffic: the kernels'
# definitions and their launch configuration (the gradient's launches live
# apart, so that changing them leaves the forward records valid).
CSRC = os.path.join(ROOT, "paper_2505_18698_amd", "csrc")
FWD_SOURCES = ("ma_kernels.hpp", "grouped.hpp", "dispatch.hpp")
BWD_SOURCES = ("backward.hpp", "dispatch_bwd.hpp", "ma_kernels.hpp", "grouped.hpp", "dispatch.hpp")


def kernel_sources_sha(kernel):
    import hashlib

    files = BWD_SOURCES if kernel in ("l_bwd", "r_bwd") else FWD_SOURCES
    src = b"".join(open(os.path.join(CSRC, f), "rb").read() for f in files)
    return hashlib.sha256(src).hexdigest()[:16]


def measured_traffic(kernel, workload):
    """HBM bytes (read + write) per launch from the committed rocprofv3 byte counters
    (profiles/traffic.json), or None when the kernel's sources changed since they
    were taken (or it was not profiled on this workload)."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        return None
    base = kernel.split("[")[0]
    k = rec.get("kernels", {}).get(f"{kernel}@{workload}")
    if k is None or k.get("source_sha256_16") != kernel_sources_sha(base):
        return None
    return k["read_bytes"] + k["write_bytes"]


def roofline_of(kernel, dtype, workload=None):
    t = kernel["avg_us"] * 1e-6
    hbm_t = kernel["alg_bytes"] / (HBM_PEAK_GBS * 1e9)
    mfma_t = kernel["alg_flops"] / (MFMA_PEAK_TFLOPS[dtype] * 1e12)
    if hbm_t >= mfma_t:
        achieved = kernel["alg_bytes"] / t / 1e9
        return {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": measured_traffic(kernel["kernel"], workload),
                "kernel": kernel["kernel"], "alg_bytes": kernel["alg_bytes"]}
    achieved = kernel["alg_flops"] / t / 1e12
    peak = MFMA_PEAK_TFLOPS[dtype]
    return {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
            "frac": round(achieved / peak, 4), "traffic": measured_traffic(kernel["kernel"], workload),
            "kernel": kernel["kernel"], "alg_flops": kernel["alg_flops"]}


def call_roofline(w, ms):
    compulsory, flops = call_work(w)
    t = ms * 1e-3
    t_hbm = compulsory / (HBM_PEAK_GBS * 1e9)
    t_mfma = flops / (MFMA_PEAK_TFLOPS[w.dtype] * 1e12)
    return {"bound": "hbm" if t_hbm >= t_mfma else "mfma", "compulsory_bytes": compulsory, "flops": flops,
            "t_roof_us": round(max(t_hbm, t_mfma) * 1e6, 3), "frac": round(max(t_hbm, t_mfma) / t, 4),
            "GB_s": round(compulsory / t / 1e9, 1), "TFLOP_s": round(flops / t / 1e12, 2)}


def cpu_baseline(w, budget_s=10.0, max_runs=20):
    import oracle
    import synth_inputs as si

    oracle.build(force=False)
    q, k, v, _ = si.make_qkv(w)
    threads = oracle.max_threads()
    runs, t0 = 0, time.time()
    while True:
        oracle.monarch_attention(q, k, v, w.m, w.b, w.T)
        runs += 1
        el = time.time() - t0
        if el >= budget_s or runs >= max_runs:
            break
    rate = runs * w.B * w.H * w.N / el
    res = {"value": round(rate, 1), "unit": UNIT, "cores": threads, "kind": "oracle",
           "sample": f"{runs} full forward passes of {w.name} (all {w.B * w.H} heads), fp64, {el:.1f}s"}
    # one thread on a bounded ViT-B/16 sample (48 of its 384 heads), for scaling context
    v = si.WORKLOADS["vit_b16_n196"]
    q1, k1, v1, _ = si.make_qkv(v.with_(B=4))
    runs1, t1 = 0, time.time()
    while True:
        oracle.monarch_attention(q1, k1, v1, v.m, v.b, v.T, threads=1)
        runs1 += 1
        el1 = time.time() - t1
        if el1 >= budget_s / 2 or runs1 >= max_runs:
            break
    res["single_thread"] = {"value": round(runs1 * 4 * v.H * v.N / el1, 1), "unit": UNIT, "cores": 1,
                            "sample": f"{runs1} passes of {v.name} at B=4 (48 heads), fp64, 1 thread, {el1:.1f}s"}
    return res


def copy_sweep(torch, sizes_mb, steps, warmup):
    """Device-to-device copies of known size (read + write = 2 x size bytes)."""
    for mb in sizes_mb:
        n = int(mb * (1 << 20)) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        warm_up(torch, lambda i: dst.copy_(src), warmup)
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record()
        for _ in range(steps):
            dst.copy_(src)
        end.record()
        end.synchronize()
        ms = start.elapsed_time(end) / steps
        print(json.dumps({"copy_mb": mb, "bytes_moved": 2 * n * 4, "us": round(ms * 1e3, 3),
                          "GB_s": round(2 * n * 4 / (ms * 1e-3) / 1e9, 1)}), flush=True)
        del src, dst


def call_traffic(w, kernels):
    """Measured HBM bytes of one call: the sum over its launches of the
    committed rocprofv3 byte counters, or None unless every launch has a
    record taken with its current sources."""
    tot = 0
    for k in kernels:
        t = measured_traffic(k["kernel"], w.name)
        if t is None:
            return None
        tot += t
    return tot


def headline_roofline(w, ms, kernels, peaks):
    """The roofline of the call: the compulsory bytes 4 N d s per head (Q, K,
    V in, O out) or the method's flops, whichever bounds it, over the call
    time.  The dominant kernel's figure on the bytes of the paper's state
    organisation (design IO) is kept beside it as a secondary field."""
    compulsory, flops = call_work(w)
    t = ms * 1e-3
    t_hbm = compulsory / (HBM_PEAK_GBS * 1e9)
    t_mfma = flops / (MFMA_PEAK_TFLOPS[w.dtype] * 1e12)
    if t_hbm >= t_mfma:
        achieved = compulsory / t / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4)}
    else:
        achieved = flops / t / 1e12
        peak = MFMA_PEAK_TFLOPS[w.dtype]
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4)}
    roof["traffic"] = call_traffic(w, kernels)
    roof["scope"] = "call"
    roof["alg_bytes"] = compulsory
    roof["alg_flops"] = flops
    if peaks:
        key = "copy_GB_s" if roof["unit"] == "GB/s" else "gemm_bf16_TFLOP_s"
        roof["frac_of_measured"] = round(roof["achieved"] / peaks[key], 4)
    dom = max(kernels, key=lambda x: x["avg_us"])
    dk = roofline_of(dom, w.dtype, w.name)
    roof["dominant_kernel"] = {"kernel": dom["kernel"], "avg_us": dom["avg_us"], "launches": len(kernels),
                               "design_io_frac": dk["frac"], "design_io_bound": dk["bound"]}
    return roof


def compact_record(w, value, ms, steps, warmup, cfg, roof, also_short):
    """The headline record (the last stdout line, with cpu_baseline and the
    details file name added by main)."""
    return {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": UNIT,
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(ms, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": cfg,
        "roofline": roof,
        "also": also_short,
    }


def record_line(result):
    """One compact JSON line, under the 4 KB a log tail keeps whole."""
    line = json.dumps(result, separators=(",", ":"))
    assert len(line) < 4096, len(line)
    return line


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="speed_n16384")
    ap.add_argument("--d", type=int, default=None, help="override the head dimension")
    ap.add_argument("--T", type=int, default=None, help="override the number of steps T")
    ap.add_argument("--also", default="speed_n4096,vit_b16_n196,speed_n4096_t3,vit_b16_n197,roberta_n1024",
                    help="comma-separated extra workloads ('' for none)")
    ap.add_argument("--backward", default="speed_n16384,speed_n4096,vit_b16_n197,sweep_n16384_d128",
                    help="comma-separated workloads for the gradient timing ('' for none)")
    ap.add_argument("--sweep", default=",".join(f"sweep_n{n}_d{d}" for n in (256, 1024, 4096, 16384)
                                                   for d in (64, 128)),
                    help="comma-separated workloads of the N / d sweep ('' for none)")
    ap.add_argument("--varlen", default="roberta_n384_b48",
                    help="comma-separated workloads timed as padded batches with per-sequence lengths ('' for none)")
    ap.add_argument("--sdpa", action="store_true",
                    help="also time torch's fused attention on the sweep shapes (context only)")
    ap.add_argument("--no-measured-peaks", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-quality", action="store_true",
                    help="skip the approximation-quality figures (error against exact attention, objective gap)")
    ap.add_argument("--details", default="bench_details.json",
                    help="file for the full record (per-kernel times, sweep, gradient, padded batches, quality); "
                         "'' for none")
    ap.add_argument("--copy-mb", type=str, default=None,
                    help="instead of the benchmark: time torch's device copy at these sizes (MB, comma "
                         "separated); the reference kernel for scaling HBM byte counters")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}, WORLD_SIZE {world}); "
              "the forward pass is not sharded across GPUs (heads would split across them with no communication).", file=sys.stderr)
        sys.exit(2)

    import torch

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    lib = os.path.join(ROOT, "paper_2505_18698_amd", "libmonarch_attn.so")
    if not os.path.exists(lib):
        import __graft_entry__

        __graft_entry__.build()
    if args.copy_mb:
        copy_sweep(torch, [float(x) for x in args.copy_mb.split(",")], args.steps, args.warmup)
        return

    import paper_2505_18698_amd as ma
    import synth_inputs as si

    w = si.WORKLOADS[args.workload]
    if args.d:
        w = w.with_(d=args.d)
    if args.T:
        w = w.with_(T=args.T)

    peaks = measured_peaks(torch) if not args.no_measured_peaks else None
    ms, kernels, meta, nsets, extra = measure(ma, torch, w, args.steps, args.warmup)
    value = w.B * w.H * w.N / (ms * 1e-3)
    cfg = {"workload": w.name, "B": w.B, "H": w.H, "N": w.N, "m": w.m, "b": w.b, "d": w.d, "T": w.T,
           "inputs": w.recipe, "alpha": meta.get("alpha"), "rotating_input_sets": nsets}
    roof = headline_roofline(w, ms, kernels, peaks)
    details = {"headline": {"config": w.describe(), "ms_per_step": ms, "kernels": kernels, **extra,
                            "roofline": roof, "call_roofline": call_roofline(w, ms)},
               "measured_peaks": peaks}
    also, also_short = [], []
    for name in [x for x in args.also.split(",") if x]:
        w2 = si.WORKLOADS[name]
        ms2, kern2, meta2, nsets2, extra2 = measure(ma, torch, w2, args.steps, args.warmup)
        r2 = headline_roofline(w2, ms2, kern2, peaks)
        cfg2 = w2.describe()
        cfg2.update({"alpha": meta2.get("alpha"), "rotating_input_sets": nsets2})
        also.append({"config": cfg2, "value": round(w2.B * w2.H * w2.N / (ms2 * 1e-3), 1), "unit": UNIT,
                     "ms_per_step": round(ms2, 6), "roofline": r2, "kernels": kern2, **extra2})
        also_short.append({"workload": name, "value": round(w2.B * w2.H * w2.N / (ms2 * 1e-3), 1),
                           "ms_per_step": round(ms2, 6), "roofline_frac": r2["frac"], "bound": r2["bound"]})
    details["also"] = also
    sweep = []
    for name in [x for x in args.sweep.split(",") if x]:
        w3 = si.WORKLOADS[name]
        ms3, kern3, meta3, _, extra3 = measure(ma, torch, w3, args.steps, args.warmup)
        rec = {"workload": name, "N": w3.N, "d": w3.d, "T": w3.T, "alpha": meta3.get("alpha"),
               "value": round(w3.B * w3.H * w3.N / (ms3 * 1e-3), 1), "ms_per_step": round(ms3, 6),
               "roofline": headline_roofline(w3, ms3, kern3, peaks), "kernels": kern3, **extra3}
        if args.sdpa and w3.d == 64 and w3.N in PAPER_SPEEDUP_VS_FA2:
            rec["context_vs_torch_sdpa"] = sdpa_context(ma, torch, w3, args.steps, args.warmup, ms3)
        sweep.append(rec)
    details["sweep"] = sweep
    details["backward"] = [measure_backward(ma, torch, si.WORKLOADS[name], args.steps, args.warmup)
                           for name in [x for x in args.backward.split(",") if x]]
    details["varlen"] = [measure_varlen(ma, torch, si.WORKLOADS[name], args.steps, args.warmup)
                         for name in [x for x in args.varlen.split(",") if x]]
    if not args.no_quality:
        details["quality"] = [quality(ma, torch, si.WORKLOADS[name]) for name in QUALITY_WORKLOADS]
    result = compact_record(w, value, ms, args.steps, args.warmup, cfg, roof, also_short)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w)
    if args.details:
        details["result"] = result
        with open(args.details, "w") as f:
            json.dump(details, f, indent=1)
        result["details"] = args.details
    print(record_line(result), flush=True)


if __name__ == "__main__":
    main()
