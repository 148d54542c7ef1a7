"""Benchmark of the ISPA hot path on one MI355X.

One step is one layer's warmup (T_warm = 12 latent frames = 4 chunks, Sec. 4.1)
at the Wan-1.3B shape (12 heads x 128, d = 1536, chunk = 4680 queries): for
each of the 4 chunks (distinct seeded inputs)

  1. F-Layer attention, dual stream: full cache of 7 chunks (32760 keys) and
     the local window of 2 chunks (9360 keys) from one pass;
  2. L-Layer attention over the local window only;
  3. statistics of the chunk: R = bf16(A_full - A_loc), G += X^T X,
     C += X^T R with X = bf16(A_loc) (4680 rows);

then, once, 4. the closed-form solve dW = (G + 1e-3 I)^-1 C (d = 1536) over
the 18720 accumulated rows, as the method solves once per layer at the end of
its warmup (Sec. 3.2). The statistics restart at the next step (the next layer).

Inputs are seeded synthetic N(0, 1) bf16 tensors already resident in HBM.
`value` is the algorithmic TFLOP/s of the whole step (visible keys only for
attention, the symmetric half of X^T X, D^3/3 + 2 D^2 D_out for the solve)
divided by the measured step time. The roofline object covers the dominant
call (the dual-stream attention: its kernel and, when the work is split over
the chip, the merge kernel), timed with HIP events on the stream it runs on.
`cpu_baseline` times the CPU oracle on a bounded sample of the same step.
The default run also times the same step at the 14B-like shape (40 heads x 128,
98280 keys; `breakdown_14b`, with its own sampled CPU baseline on 4 of the 40
heads) and, at both shapes, the dual-stream call against a single-stream call
over the full cache (`dual_overhead`: the cost of also writing the local result,
Sec. 3.4). `--workload 14b` runs the 14B-like shape alone; `--workload rollout`
the 60-chunk streaming rollout.
"""

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import torch  # noqa: E402

WORKLOADS = {
    "1.3b": dict(name="wan1.3b-layer-warmup-step", heads=12, head_dim=128, n_q=4680, cache_len=32760,
                 window=9360, sink=0, lam=1e-3, t_warm_chunks=4, n_layers=30),
    "14b": dict(name="14b-layer-warmup-step", heads=40, head_dim=128, n_q=4680, cache_len=98280,
                window=9360, sink=0, lam=1e-3, t_warm_chunks=4, n_layers=40),
}

# the long streaming rollout at the 1.3B shape: 30 layers, half of them
# L-Layers holding a window of 2 chunks, 60 chunks of 4680 queries
ROLLOUT = dict(name="wan1.3b-rollout-60-chunks", heads=12, head_dim=128, n_q=4680, chunks=60, layers=30,
               l_layers=15, window=9360, sink=0)
KV_BYTES_PER_KEY = 2 * 2  # one bf16 key and one bf16 value element per hidden unit

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA (published)
PEAK_INT8_TOPS = 5000.0    # MI355X dense int8 MFMA
PEAK_FP32_TFLOPS = 157.3   # MI355X fp32 matrix / vector (published)
PEAK_HBM_GBS = 8000.0

# HBM bytes of one dual-stream attention call (one launch of the attention
# kernel; neither shape splits its work items), from rocprofv3 FETCH_SIZE and WRITE_SIZE
# scaled by the plain-copy calibration (profiles/attn_fast_wan13b_dual.md,
# profiles/hbm_copy_calibration.md). Valid only for the kernel source they were
# taken on; reported as null otherwise.
MEASURED_TRAFFIC = {
    "1.3b": {"attn_chunk_sha256_16": "b262289ba401158f", "bytes_per_launch": 391.7e6},
    "14b": {"attn_chunk_sha256_16": "b262289ba401158f", "bytes_per_launch": 3059.9e6},
}


def attn_source_hash():
    """sha256[:16] over the sources of the attention launch (the C++ kernels and
    merge, the generator of the head_dim-128 assembly kernel and its host side)."""
    import hashlib
    h = hashlib.sha256()
    for name in ("attn_chunk.hip", "attn_fast_gen.py", "attn_fast.cpp"):
        with open(os.path.join(ROOT, "paper_2607_00712_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def flops(w):
    D = w["heads"] * w["head_dim"]
    n_q, N, win = w["n_q"], w["cache_len"], w["window"]
    vis_local = min(N, win + min(w["sink"], N))
    f = {
        "attn_dual": 4.0 * n_q * N * D,
        "attn_local": 4.0 * n_q * vis_local * D,
        "gram": float(n_q) * D * (D + 1) + 2.0 * n_q * D * D,
        "solve": D ** 3 / 3.0 + 2.0 * D * D * D,
    }
    return f


def step_flops(w, f, only="all"):
    """Algorithmic flop of one step: T_warm chunks of attention and statistics,
    one solve (with `only`, of that part alone)."""
    per_chunk = {"attn_dual": f["attn_dual"], "attn_local": f["attn_local"], "accum_stats": f["gram"]}
    total = 0.0
    for part, fl in per_chunk.items():
        if only in ("all", part):
            total += w["t_warm_chunks"] * fl
    if only in ("all", "solve"):
        total += f["solve"]
    return total


def gpu_run(w, steps, warmup, only="all", extras=True):
    """Times `steps` layer warmups. Returns the wall-clock ms per step and the
    per-part averages: ms per call for the attention calls and the statistics
    (one per chunk), ms per solve."""
    import synth
    import paper_2607_00712_amd as ispa

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    H, d = w["heads"], w["head_dim"]
    D = H * d
    n_chunks = w["t_warm_chunks"]
    chunks = [synth.chunk_qkv(2607, 0, c, w["n_q"], w["cache_len"], D, dev) for c in range(n_chunks)]
    out = torch.empty((w["n_q"], D), dtype=torch.float32, device=dev)
    out_l = torch.empty_like(out)
    out_L = torch.empty_like(out)
    lse = torch.empty((H, w["n_q"]), dtype=torch.float32, device=dev)
    lse_l = torch.empty_like(lse)
    lse_L = torch.empty_like(lse)
    stats = ispa.Stats(D, D, max_rows=w["n_q"], device=dev)
    dw = torch.empty((D, D), dtype=torch.float32, device=dev)
    eps_dev = torch.zeros((1,), dtype=torch.float64, device=dev)
    status_dev = torch.zeros((1,), dtype=torch.int32, device=dev)

    run = {p: only in ("all", p) for p in ("attn_dual", "attn_local", "accum_stats", "solve")}
    names = ("attn_dual", "attn_local", "accum_stats")

    def step(ev=None):
        # ev: per chunk 4 events around the three parts, then 1 after the solve
        stats.reset()
        for c, (q, k, v) in enumerate(chunks):
            if ev is not None:
                ev[3 * c].record()
            if run["attn_dual"]:
                ispa.attn_chunk(q, k, v, w["cache_len"], w["window"], H, sink_len=w["sink"], dual=True,
                                out=out, lse=lse, out_local=out_l, lse_local=lse_l)
            if ev is not None:
                ev[3 * c + 1].record()
            if run["attn_local"]:
                ispa.attn_chunk(q, k, v, w["cache_len"], w["window"], H, sink_len=w["sink"],
                                out=out_L, lse=lse_L)
            if ev is not None:
                ev[3 * c + 2].record()
            if run["accum_stats"]:
                stats.accum(out_l, out, out_l)
        if ev is not None:
            ev[3 * n_chunks].record()
        if run["solve"]:
            # the solve that does not wait: eps and the status word stay in
            # device memory (a warmup reads the scores of all layers at once
            # for the ranking); checked once after the timed steps
            stats.solve_async(w["lam"], delta_w=dw, eps=eps_dev, status=status_dev)
        if ev is not None:
            ev[3 * n_chunks + 1].record()

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    n_ev = 3 * n_chunks + 2
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(n_ev)] for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        step(events[i])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    parts = {"attn_dual": [], "attn_local": [], "accum_stats": [], "solve": []}
    for ev in events:
        for c in range(n_chunks):
            for j, name in enumerate(names):
                parts[name].append(ev[3 * c + j].elapsed_time(ev[3 * c + j + 1]))
        parts["solve"].append(ev[3 * n_chunks].elapsed_time(ev[3 * n_chunks + 1]))
    if run["solve"]:
        if int(status_dev.item()) != 0 or not math.isfinite(float(eps_dev.item())):
            raise RuntimeError("solve: G + lambda I not positive definite in the timed steps")
    avg = {k2: sum(v2) / len(v2) for k2, v2 in parts.items()}
    ms_step = (t1 - t0) * 1e3 / steps
    if only == "all" and extras:
        avg["absorb"] = absorb_run(ispa, w, chunks[0][1], chunks[0][2], dw, dev)
        avg["solve_all_layers"] = solve_all_run(ispa, w, stats, dev)
        avg["dual_overhead"] = dual_overhead_run(ispa, w, chunks[0], dev)
        avg["attn_zero_inputs"] = zero_inputs_run(ispa, w, dev)
    return ms_step, avg


def zero_inputs_run(ispa, w, dev, reps=5):
    """Diagnostic beside the step (not part of it): the same dual-stream call
    on all-zero Q, K and V. The instruction stream, the tiles visited and the
    memory traffic are those of the real call; only the operand bits do not
    toggle. With random bf16 operands the matrix cores' power holds the chip
    below its peak clock (GRBM_GUI_ACTIVE gives about 1.75 GHz against about
    2.4 GHz for zero operands at the 14B shape), so the ratio of the two rates
    separates the power limit from the kernel's own schedule."""
    H, D = w["heads"], w["heads"] * w["head_dim"]
    N = w["cache_len"]
    q = torch.zeros((w["n_q"], D), dtype=torch.bfloat16, device=dev)
    kv = torch.zeros((N, D), dtype=torch.bfloat16, device=dev)
    out = torch.empty((w["n_q"], D), dtype=torch.float32, device=dev)
    out_l = torch.empty_like(out)
    lse = torch.empty((H, w["n_q"]), dtype=torch.float32, device=dev)
    lse_l = torch.empty_like(lse)
    call = lambda: ispa.attn_chunk(q, kv, kv, N, w["window"], H, sink_len=w["sink"], dual=True,
                                   out=out, lse=lse, out_local=out_l, lse_local=lse_l)
    for _ in range(6):
        call()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        call()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del q, kv
    fl = flops(w)["attn_dual"]
    return {"attn_dual_ms": round(ms, 4), "attn_dual_tflops": round(fl / ms / 1e9, 1),
            "frac": round(fl / ms / 1e9 / PEAK_BF16_TFLOPS, 4),
            "what": "diagnostic: the dual call on all-zero inputs (same instructions and traffic, no operand "
                    "toggling, so the clock is not power-limited); mean of %d back-to-back calls" % reps}


def dual_overhead_run(ispa, w, qkv, dev, reps=20):
    """The dual-stream call (full and local results from one pass) against a
    single-stream call over the same full cache (an F-Layer), on the same
    inputs. The two calls alternate back to back on the stream (no host
    synchronisation between them, so both see the same clock and power
    state); each is bracketed by HIP events and the medians of `reps`
    timings are compared. Sec. 3.4 puts the cost of the LSE fusion below one
    percent of the run time."""
    q, k, v = qkv
    H = w["heads"]
    N = w["cache_len"]
    out = torch.empty((w["n_q"], H * w["head_dim"]), dtype=torch.float32, device=dev)
    out_l = torch.empty_like(out)
    lse = torch.empty((H, w["n_q"]), dtype=torch.float32, device=dev)
    lse_l = torch.empty_like(lse)
    dual = lambda: ispa.attn_chunk(q, k, v, N, w["window"], H, sink_len=w["sink"], dual=True,
                                   out=out, lse=lse, out_local=out_l, lse_local=lse_l)
    full = lambda: ispa.attn_chunk(q, k, v, N, N, H, out=out, lse=lse)
    for _ in range(3):
        dual()
        full()
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(reps)]
    for e in ev:
        e[0].record()
        dual()
        e[1].record()
        e[2].record()
        full()
        e[3].record()
    torch.cuda.synchronize()
    t_dual = sorted(e[0].elapsed_time(e[1]) for e in ev)[reps // 2]
    t_full = sorted(e[2].elapsed_time(e[3]) for e in ev)[reps // 2]
    return {"dual_ms": round(t_dual, 4), "full_single_ms": round(t_full, 4),
            "overhead": round(t_dual / t_full - 1.0, 4),
            "what": "dual-stream call (full + local outputs) / single-stream full-cache call - 1, same inputs, "
                    "the two calls alternating back to back, median of %d HIP-event timings each" % reps}


def absorb_run(ispa, w, k, v, dw, dev, reps=10):
    """The one-off absorption at the end of warmup (Sec. 3.3), outside the step:
    the in-place update of a bf16 linear-layer weight with dW^T, and the
    eviction of the layer's cache to its local set. Returns ms and HBM GB/s."""
    D = w["heads"] * w["head_dim"]
    weight = torch.zeros((D, D), dtype=torch.bfloat16, device=dev)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    inj = timed(lambda: ispa.inject_modulation(weight, dw, transposed=True))
    ring = (torch.empty((w["sink"] + w["window"], D), dtype=torch.bfloat16, device=dev),
            torch.empty((w["sink"] + w["window"], D), dtype=torch.bfloat16, device=dev))
    ev = timed(lambda: ispa.LocalKV(k, v, w["cache_len"], w["window"], w["sink"], ring=ring))
    rows = ispa.LocalKV(k, v, w["cache_len"], w["window"], w["sink"], ring=ring).rows
    # the L-Layer's output projection of one chunk with the modulated weight
    a = k[: w["n_q"]]
    y = torch.empty((w["n_q"], D), dtype=torch.bfloat16, device=dev)
    pj = timed(lambda: ispa.project(a, weight, out=y))
    # its W8A8 form (Sec. 4): per-token codes of the chunk's activations, then
    # the int8 projection with per-channel weight codes
    qa = torch.empty((w["n_q"], D), dtype=torch.int8, device=dev)
    sa = torch.empty((w["n_q"],), dtype=torch.float32, device=dev)
    qw, sw = ispa.quantize_rows(weight)
    qt = timed(lambda: ispa.quantize_rows(a, q=qa, scale=sa))
    pj8 = timed(lambda: ispa.project_w8a8(qa, sa, qw, sw, out=y))
    inj_bytes = D * D * (2 + 4 + 2)
    ev_bytes = rows * D * 2 * 2 * 2
    pj_flop = 2.0 * w["n_q"] * D * D
    return {"inject_ms": round(inj, 4), "inject_gbs": round(inj_bytes / inj / 1e6, 1),
            "evict_ms": round(ev, 4), "evict_gbs": round(ev_bytes / ev / 1e6, 1),
            "hbm_peak_gbs": PEAK_HBM_GBS,
            "project_ms": round(pj, 4), "project_tflops": round(pj_flop / pj / 1e9, 1),
            "project_frac": round(pj_flop / pj / 1e9 / PEAK_BF16_TFLOPS, 4),
            "quantize_ms": round(qt, 4), "quantize_gbs": round(w["n_q"] * D * (2 + 1) / qt / 1e6, 1),
            "project_w8a8_ms": round(pj8, 4), "project_w8a8_tops": round(pj_flop / pj8 / 1e9, 1),
            "project_w8a8_frac": round(pj_flop / pj8 / 1e9 / PEAK_INT8_TOPS, 4)}


def project_run(w, steps, warmup):
    """The chunk's output projection alone (`--only project`, for profiling):
    A [n_q, D] W^T with random bf16 operands, then its W8A8 form on the codes
    of the same operands; mean of `steps` calls each after `warmup`."""
    import paper_2607_00712_amd as ispa
    dev = torch.device("cuda", 0)
    D, n = w["heads"] * w["head_dim"], w["n_q"]
    g = torch.Generator(device=dev).manual_seed(11)
    a = torch.randn((n, D), device=dev, generator=g).to(torch.bfloat16)
    weight = (torch.randn((D, D), device=dev, generator=g) / D ** 0.5).to(torch.bfloat16)
    y = torch.empty((n, D), dtype=torch.bfloat16, device=dev)
    qa, sa = ispa.quantize_rows(a)
    qw, sw = ispa.quantize_rows(weight)

    def timed(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    pj = timed(lambda: ispa.project(a, weight, out=y))
    pj8 = timed(lambda: ispa.project_w8a8(qa, sa, qw, sw, out=y))
    fl = 2.0 * n * D * D
    return {"only": "project", "workload": w["name"], "shape": [n, D, D],
            "project_ms": round(pj, 4), "project_tflops": round(fl / pj / 1e9, 1),
            "project_frac": round(fl / pj / 1e9 / PEAK_BF16_TFLOPS, 4),
            "project_w8a8_ms": round(pj8, 4), "project_w8a8_tops": round(fl / pj8 / 1e9, 1),
            "project_w8a8_frac": round(fl / pj8 / 1e9 / PEAK_INT8_TOPS, 4)}


def solve_all_run(ispa, w, stats, dev, reps=3):
    """The end of warmup solves every layer (Sec. 3.3, the eps ranking needs
    all of them): n_layers systems of the step's size (copies of the step's
    G, C and ||R||^2) by one batched call (ispa_solve_modulation_batch) and by
    one call per layer, timed with HIP events."""
    D = w["heads"] * w["head_dim"]
    n = w["n_layers"]
    G, C, S, _ = stats.views()
    sb = ispa.StatsBatch(n, D, D, max_rows=1, device=dev)
    for st in sb.layers:
        g, c, s, _ = st.views()
        g.copy_(G)
        c.copy_(C)
        s.copy_(S)
    dw = torch.empty((n, D, D), dtype=torch.float32, device=dev)
    eps = torch.empty((n,), dtype=torch.float64, device=dev)
    status = torch.empty((n,), dtype=torch.int32, device=dev)

    def batched():
        sb.solve(w["lam"], delta_w=dw, eps=eps, status=status)

    def one_by_one():
        for i, st in enumerate(sb.layers):
            st.solve_async(w["lam"], delta_w=dw[i], eps=eps[i:i + 1], status=status[i:i + 1])

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        ms = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ms.append(e0.elapsed_time(e1))
        return sorted(ms)[len(ms) // 2]

    t_b = timed(batched)
    ok_b = int(status.sum().item()) == 0
    t_1 = timed(one_by_one)
    ok_1 = int(status.sum().item()) == 0
    sb.close()
    del sb
    if not (ok_b and ok_1):
        raise RuntimeError("solve of all layers: G + lambda I not positive definite")
    flop = n * (D ** 3 / 3.0 + 2.0 * D * D * D)
    return {"layers": n, "batched_ms": round(t_b, 3), "one_by_one_ms": round(t_1, 3),
            "speedup": round(t_1 / t_b, 3), "batched_tflops": round(flop / t_b / 1e9, 2),
            "batched_frac_fp32_peak": round(flop / t_b / 1e9 / 157.3, 4),
            "one_by_one_tflops": round(flop / t_1 / 1e9, 2)}


def discrepancy_rotating(w, steps, warmup, sets=8):
    """accum_stats over `sets` distinct (y_full, y_local) fp32 chunk pairs used
    in rotation (8 x 57.5 MB = 460 MB at the 1.3B width, more than the 256 MB
    last-level cache), so that the discrepancy kernel's reads come from HBM;
    x aliases y_local as in the warmup chain. For a kernel trace of the
    discrepancy and Gram kernels on an HBM-resident working set."""
    import synth
    import paper_2607_00712_amd as ispa
    dev = torch.device("cuda", 0)
    D = w["heads"] * w["head_dim"]
    ys = [(synth.normal((w["n_q"], D), synth.seed_of(2607, i, synth.Y_FULL), dev, dtype=torch.float32),
           synth.normal((w["n_q"], D), synth.seed_of(2607, i, synth.Y_LOCAL), dev, dtype=torch.float32))
          for i in range(sets)]
    st = ispa.Stats(D, D, max_rows=w["n_q"], device=dev)
    for i in range(warmup):
        yf, yl = ys[i % sets]
        st.accum(yl, yf, yl)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(steps):
        yf, yl = ys[i % sets]
        st.accum(yl, yf, yl)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    per_call_bytes = w["n_q"] * D * (4 + 4 + 2 + 2)
    return {"only": "discrepancy_rotating", "workload": w["name"], "sets": sets,
            "working_set_mb": round(sets * 2 * w["n_q"] * D * 4 / 1e6, 1), "accum_stats_ms": round(ms, 4),
            "discrepancy_bytes_per_call": per_call_bytes}


def hbm_copy(steps, warmup, nbytes=1 << 30):
    """A plain 1 GiB device-to-device copy (torch's copy kernel), the yardstick
    for the HBM byte counters: FETCH_SIZE / WRITE_SIZE of this copy against the
    known 1 GiB read and 1 GiB written give the counters' scale."""
    dev = torch.device("cuda", 0)
    src = torch.empty(nbytes, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    for _ in range(warmup):
        dst.copy_(src)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        dst.copy_(src)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    return {"only": "hbm_copy", "bytes_read": nbytes, "bytes_written": nbytes, "ms": round(ms, 4),
            "GB/s": round(2 * nbytes / ms / 1e6, 1)}


def lib_ref(steps, warmup):
    """Library references on the same shapes, for context beside the kernels
    here (never part of the step): torch's scaled-dot-product attention limited
    to its flash backend (bf16, one output per call: the full cache and the
    window timed separately), torch's bf16 GEMM for X^T R, torch's fp32
    Cholesky factor plus triangular solves for one ridge system, and torch's
    bf16 GEMM for the chunk's projection A W^T. Inputs are random; each entry is
    the mean of `steps` calls after `warmup`, timed with events on torch's
    stream."""
    from torch.nn.attention import SDPBackend, sdpa_kernel
    import torch.nn.functional as F
    dev = torch.device("cuda", 0)
    g = torch.Generator(device=dev).manual_seed(7)

    def timed(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    out = {"only": "lib_ref", "steps": steps, "warmup": warmup}
    for key in ("1.3b", "14b"):
        w = WORKLOADS[key]
        H, hd, n_q, N, win = w["heads"], w["head_dim"], w["n_q"], w["cache_len"], w["window"]
        D = H * hd
        r = {}
        q = torch.randn(1, H, n_q, hd, device=dev, dtype=torch.bfloat16, generator=g)
        k = torch.randn(1, H, N, hd, device=dev, dtype=torch.bfloat16, generator=g)
        v = torch.randn(1, H, N, hd, device=dev, dtype=torch.bfloat16, generator=g)
        kw, vw = k[:, :, N - win:].contiguous(), v[:, :, N - win:].contiguous()
        with sdpa_kernel([SDPBackend.FLASH_ATTENTION]):
            ms = timed(lambda: F.scaled_dot_product_attention(q, k, v))
            r["sdpa_flash_full"] = {"ms": round(ms, 4), "tflops": round(4.0 * n_q * N * D / ms / 1e9, 1)}
            ms = timed(lambda: F.scaled_dot_product_attention(q, kw, vw))
            r["sdpa_flash_window"] = {"ms": round(ms, 4), "tflops": round(4.0 * n_q * win * D / ms / 1e9, 1)}
        del q, k, v, kw, vw
        xt = torch.randn(D, n_q, device=dev, dtype=torch.bfloat16, generator=g)
        rr = torch.randn(n_q, D, device=dev, dtype=torch.bfloat16, generator=g)
        ms = timed(lambda: torch.mm(xt, rr))
        r["gemm_bf16_xtr"] = {"shape": [D, D, n_q], "ms": round(ms, 4),
                              "tflops": round(2.0 * n_q * D * D / ms / 1e9, 1)}
        wt = torch.randn(D, D, device=dev, dtype=torch.bfloat16, generator=g)
        ms = timed(lambda: torch.mm(rr, wt))
        r["gemm_bf16_proj"] = {"shape": [n_q, D, D], "ms": round(ms, 4),
                               "tflops": round(2.0 * n_q * D * D / ms / 1e9, 1)}
        del xt, rr, wt
        a = torch.randn(D, 2 * D, device=dev, dtype=torch.float32, generator=g)
        spd = a @ a.t() / (2 * D) + 1e-3 * torch.eye(D, device=dev)
        c = torch.randn(D, D, device=dev, dtype=torch.float32, generator=g)

        def chol_solve():
            fac = torch.linalg.cholesky(spd)
            return torch.cholesky_solve(c, fac)
        ms = timed(chol_solve)
        r["torch_cholesky_solve_fp32"] = {"shape": [D, D], "ms": round(ms, 4),
                                          "tflops": round((D ** 3 / 3.0 + 2.0 * D ** 3) / ms / 1e9, 2)}
        del a, spd, c
        torch.cuda.empty_cache()
        out[key] = r
    return out


def cpu_baseline(w, budget_rows=512, heads=None):
    """The oracle on a bounded sample of one step, scaled to TFLOP/s: attention
    of `budget_rows` query rows over all keys for `heads` of the heads (all by
    default), the statistics of those rows at the full width, and the full
    D x D solve; the sampled times are scaled linearly to a whole step."""
    import numpy as np
    import oracle
    import synth

    H, d = w["heads"], w["head_dim"]
    D = H * d
    hs = H if heads is None else heads
    cores = len(os.sched_getaffinity(0))
    q, k, v = synth.chunk_qkv(2607, 0, 0, w["n_q"], w["cache_len"], D, "cpu")
    rows = np.arange(budget_rows)
    # the first hs heads (columns of the hidden layout), as their own tensors
    qn = q[:, :hs * d].double().numpy()
    kn = k[:, :hs * d].double().numpy()
    vn = v[:, :hs * d].double().numpy()
    del q, k, v
    f = flops(w)
    frac = budget_rows / w["n_q"] * hs / H
    t = time.perf_counter()
    o = oracle.chunk_attention(qn, kn, vn, w["cache_len"], w["window"], hs, sink_len=w["sink"],
                               branches=("full", "local"), query_rows=rows)
    oracle.chunk_attention(qn, kn, vn, w["cache_len"], w["window"], hs, sink_len=w["sink"],
                           branches=("local",), query_rows=rows)
    t_attn = time.perf_counter() - t
    del kn, vn
    # statistics of the sampled rows at the full width D (the sampled heads'
    # outputs tiled across the hidden dimension)
    reps = H // hs
    ol = np.tile(o["local"][0], (1, reps)).astype(np.float32)
    of = np.tile(o["full"][0], (1, reps)).astype(np.float32)
    st = oracle.Stats(D, D)
    xs = oracle.bf16_round(ol)
    t = time.perf_counter()
    st.accumulate(xs, of, ol)
    t_stats = time.perf_counter() - t
    G = st.G + np.eye(D) * 10.0  # sample rows < D: keep the system well posed for timing
    t = time.perf_counter()
    oracle.solve_modulation(G, st.C, w["lam"])
    t_solve = time.perf_counter() - t
    # scale each sampled part to a whole step
    frac_rows = budget_rows / w["n_q"]
    t_step = w["t_warm_chunks"] * ((t_attn / frac) + (t_stats / frac_rows)) + t_solve
    total_flops = step_flops(w, f)
    head_txt = f"all {H} heads" if hs == H else f"{hs} of {H} heads"
    return {
        "value": total_flops / t_step / 1e12,
        "unit": "TFLOP/s",
        "cores": cores,
        "kind": "oracle",
        "sample": (f"fp64 numpy oracle: F-Layer dual + L-Layer attention for {budget_rows} of {w['n_q']} query "
                   f"rows of one chunk ({head_txt}, all {w['cache_len']} keys), statistics of those rows at "
                   f"d = {D}, full {D}x{D} Cholesky solve; attention time scaled by {w['n_q']}/{budget_rows}"
                   + ("" if hs == H else f" x {H}/{hs}") + f", statistics by {w['n_q']}/{budget_rows}, both by the "
                   f"{w['t_warm_chunks']} chunks of a step (linear extrapolation); measured "
                   f"{t_attn:.2f}s + {t_stats:.2f}s + {t_solve:.2f}s"),
        "extrapolated": True,
        "ms_per_step_extrapolated": t_step * 1e3,
    }


def rollout_run(reps=3, warmup=2):
    """Streaming rollout (60 chunks, 30 layers): per chunk, every layer gets
    fresh queries and appends its chunk of keys and values; F-Layers attend to
    their whole cache (4680 n keys at chunk n), L-Layers to the ring of their
    last 2 chunks (after the permanent eviction, Sec. 3.3). The all-F baseline
    attends every layer to its whole cache: the F-Layers' launches are shared,
    the L-Layers' full-cache launches are timed on the same keys and values.
    Returns the JSON record."""
    import synth
    import paper_2607_00712_amd as ispa

    w = ROLLOUT
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    H, n_q, win, sink = w["heads"], w["n_q"], w["window"], w["sink"]
    D = H * w["head_dim"]
    n_layers, n_l = w["layers"], w["l_layers"]
    n_f = n_layers - n_l
    cap = n_q * w["chunks"]
    # full caches of every layer (an L-Layer's one only feeds the baseline and
    # its own ring), and the L-Layers' rings of sink + window rows
    kc = [torch.empty((cap, D), dtype=torch.bfloat16, device=dev) for _ in range(n_layers)]
    vc = [torch.empty((cap, D), dtype=torch.bfloat16, device=dev) for _ in range(n_layers)]
    rings = [(torch.empty((sink + win, D), dtype=torch.bfloat16, device=dev),
              torch.empty((sink + win, D), dtype=torch.bfloat16, device=dev)) for _ in range(n_l)]
    local = [None] * n_l
    out = torch.empty((n_q, D), dtype=torch.float32, device=dev)
    lse = torch.empty((H, n_q), dtype=torch.float32, device=dev)
    per_key_layer = D * KV_BYTES_PER_KEY
    res = {"chunk": [], "keys_f": [], "keys_l": [], "ispa_ms": [], "f_layers_ms": [], "l_layers_ms": [],
           "all_f_ms": [], "kv_gb_ispa": [], "kv_gb_all_f": []}
    fl_ispa = fl_allf = t_ispa = t_allf = 0.0
    t_f60 = None
    for n in range(1, w["chunks"] + 1):
        N = n_q * n
        qs = []
        for layer in range(n_layers):
            q, kn, vn = synth.rollout_chunk(layer, n, n_q, D, dev)
            qs.append(q)
            kc[layer][N - n_q:N].copy_(kn)
            vc[layer][N - n_q:N].copy_(vn)
            if layer >= n_f:
                j = layer - n_f
                if local[j] is None:
                    local[j] = ispa.LocalKV(kc[layer], vc[layer], N, win, sink, ring=rings[j])
                else:
                    local[j].append(kn, vn)
        torch.cuda.synchronize()

        def f_layers():
            for layer in range(n_f):
                ispa.attn_chunk(qs[layer], kc[layer], vc[layer], N, N, H, out=out, lse=lse)

        def l_layers():
            for j in range(n_l):
                r = local[j].rows
                ispa.attn_chunk(qs[n_f + j], local[j].k, local[j].v, r, r, H, out=out, lse=lse)

        def l_as_f():
            for layer in range(n_f, n_layers):
                ispa.attn_chunk(qs[layer], kc[layer], vc[layer], N, N, H, out=out, lse=lse)

        for _ in range(warmup if n == 1 else 0):
            f_layers(); l_layers(); l_as_f()
        samples = []
        for _ in range(reps):
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
            ev[0].record(); f_layers(); ev[1].record(); l_layers(); ev[2].record(); l_as_f(); ev[3].record()
            torch.cuda.synchronize()
            samples.append([ev[i].elapsed_time(ev[i + 1]) for i in range(3)])
        tf, tl, tx = (sorted(s[i] for s in samples)[len(samples) // 2] for i in range(3))
        keys_l = min(N, win + min(sink, N))
        res["chunk"].append(n)
        res["keys_f"].append(N)
        res["keys_l"].append(keys_l)
        res["f_layers_ms"].append(round(tf, 4))
        res["l_layers_ms"].append(round(tl, 4))
        res["ispa_ms"].append(round(tf + tl, 4))
        res["all_f_ms"].append(round(tf + tx, 4))
        res["kv_gb_ispa"].append(round((n_f * N + n_l * keys_l) * per_key_layer / 1e9, 3))
        res["kv_gb_all_f"].append(round(n_layers * N * per_key_layer / 1e9, 3))
        fl_ispa += 4.0 * n_q * D * (n_f * N + n_l * keys_l)
        fl_allf += 4.0 * n_q * D * n_layers * N
        t_ispa += tf + tl
        t_allf += tf + tx
        if n == w["chunks"]:
            t_f60 = tf / n_f
        print(f"[rollout] chunk {n}: ISPA {tf + tl:.3f} ms, all-F {tf + tx:.3f} ms", file=sys.stderr, flush=True)
    f60 = 4.0 * n_q * D * n_q * w["chunks"]
    achieved = f60 / (t_f60 * 1e-3) / 1e12
    return {
        "metric": "streaming rollout attention TFLOP/s (15 F + 15 L layers, 60 chunks)",
        "value": round(fl_ispa / (t_ispa * 1e-3) / 1e12, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": w["chunks"],
        "warmup": warmup,
        "ms_per_step": round(t_ispa / w["chunks"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w["name"], "heads": H, "head_dim": w["head_dim"], "chunk_queries": n_q,
                   "layers": n_layers, "l_layers": n_l, "window": win, "sink": sink, "chunks": w["chunks"],
                   "step": "one chunk: attention of every layer (F-Layers over the whole cache, L-Layers over "
                           "their ring); median of %d timings per chunk" % reps},
        "roofline": {"kernel": "ispa_attn_fast_d128 (F-Layer, full cache of 280800 keys, chunk 60)",
                     "bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": None},
        "summary": {
            "ispa_total_ms": round(t_ispa, 2), "all_f_total_ms": round(t_allf, 2),
            "speedup_total": round(t_allf / t_ispa, 4),
            "speedup_chunk60": round(res["all_f_ms"][-1] / res["ispa_ms"][-1], 4),
            "flop_ispa": fl_ispa, "flop_all_f": fl_allf,
            "all_f_tflops": round(fl_allf / (t_allf * 1e-3) / 1e12, 2),
            "kv_ratio_chunk60": round(res["kv_gb_ispa"][-1] / res["kv_gb_all_f"][-1], 4),
        },
        "per_chunk": res,
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", choices=sorted(WORKLOADS) + ["rollout"], default="1.3b",
                    help="1.3b / 14b: one warmup step of one layer; rollout: the 60-chunk streaming "
                         "rollout of 30 layers (per-chunk attention time and KV bytes against all F-Layers)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--step-only", action="store_true",
                    help="skip the measurements after the timed steps (absorption kernels, the solve of all "
                         "layers), e.g. for a kernel trace of the step alone")
    ap.add_argument("--no-14b", action="store_true",
                    help="skip the 14B-shaped step that the default 1.3B run also times (breakdown_14b)")
    ap.add_argument("--only", choices=["all", "attn_dual", "attn_local", "accum_stats", "solve", "hbm_copy",
                                       "discrepancy", "lib_ref", "project", "attn_zero"],
                    default="all",
                    help="time one part of the step alone (for profiling); the JSON line then covers that part")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the ISPA hot path here has no multi-GPU "
              "path (heads or layers would shard with no exchange).", file=sys.stderr)
        sys.exit(2)
    if args.only == "hbm_copy":
        print(json.dumps(hbm_copy(args.steps, args.warmup)), flush=True)
        return
    if args.only == "project":
        print(json.dumps(project_run(WORKLOADS[args.workload], args.steps, args.warmup)), flush=True)
        return
    if args.only == "attn_zero":
        # the dual call on all-zero inputs alone (for counters beside --only attn_dual)
        import paper_2607_00712_amd as ispa
        dev = torch.device("cuda", 0)
        torch.cuda.set_device(dev)
        rec = zero_inputs_run(ispa, WORKLOADS[args.workload], dev, reps=args.steps)
        rec.update({"only": "attn_zero", "workload": args.workload, "steps": args.steps})
        print(json.dumps(rec), flush=True)
        return
    if args.only == "lib_ref":
        print(json.dumps(lib_ref(args.steps, args.warmup)), flush=True)
        return
    if args.only == "discrepancy":
        print(json.dumps(discrepancy_rotating(WORKLOADS[args.workload], args.steps, args.warmup)), flush=True)
        return
    if args.workload == "rollout":
        print(json.dumps(rollout_run(warmup=args.warmup)), flush=True)
        return
    w = WORKLOADS[args.workload]
    f = flops(w)
    ms_step, avg = gpu_run(w, args.steps, args.warmup, args.only, extras=not args.step_only)
    total = step_flops(w, f, args.only)
    value = total / (ms_step * 1e-3) / 1e12
    attn_ms = avg["attn_dual"]
    mt = MEASURED_TRAFFIC.get(args.workload)
    traffic = mt["bytes_per_launch"] if mt and mt["attn_chunk_sha256_16"] == attn_source_hash() else None
    achieved = f["attn_dual"] / (attn_ms * 1e-3) / 1e12
    rec = {
        "metric": "chunk attention TFLOP/s (F vs L layer) + stats/solve ms, 1.3B/14B shapes",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": w["name"],
            "heads": w["heads"], "head_dim": w["head_dim"], "chunk_queries": w["n_q"],
            "cache_len": w["cache_len"], "window": w["window"], "sink": w["sink"],
            "d": w["heads"] * w["head_dim"], "lambda": w["lam"],
            "step": "one layer's warmup: 4 chunks x (F-Layer dual attention + L-Layer attention + accum_stats), "
                    "then one solve over the 18720 accumulated rows",
            "t_warm_chunks": w["t_warm_chunks"],
            "accumulate": "fp32 (attention, Gram); solve fp32",
        },
        "roofline": {
            "kernel": "ispa_attn_fast_d128 (F-Layer, dual stream; one launch per call, whole work items: "
                      "228 of them fill 89% of the chip, which at its power limit runs them as fast as split)",
            "bound": "mfma",
            "achieved": round(achieved, 2),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
            "traffic": traffic,
            "traffic_unit": "HBM bytes per call (rocprofv3 FETCH_SIZE + WRITE_SIZE of the attention kernel, "
                            "copy-calibrated)",
        },
        "breakdown": {
            "attn_dual_ms": round(avg["attn_dual"], 4),
            "attn_dual_tflops": round(f["attn_dual"] / avg["attn_dual"] / 1e9, 1),
            "attn_local_ms": round(avg["attn_local"], 4),
            "attn_local_tflops": round(f["attn_local"] / avg["attn_local"] / 1e9, 1),
            "accum_stats_ms": round(avg["accum_stats"], 4),
            "gram_tflops": round(f["gram"] / avg["accum_stats"] / 1e9, 1),
            "solve_ms": round(avg["solve"], 4),
            "solve_tflops": round(f["solve"] / avg["solve"] / 1e9, 2),
            "per": "attention and accum_stats: ms per chunk call (4 per step); solve: ms per step",
            "flop": {k2: v2 for k2, v2 in f.items()},
            "flop_step": total,
            "absorb": avg.get("absorb"),
            "solve_all_layers": avg.get("solve_all_layers"),
        },
        "dual_overhead": avg.get("dual_overhead"),
        "attn_zero_inputs": avg.get("attn_zero_inputs"),
    }
    if args.only != "all":
        rec["only"] = args.only
    if args.workload == "1.3b" and args.only == "all" and not args.no_14b:
        print("[bench] 14B-shaped step", file=sys.stderr, flush=True)
        w14 = WORKLOADS["14b"]
        steps14 = max(3, min(args.steps, 8))
        ms14, avg14 = gpu_run(w14, steps14, min(args.warmup, 2), "all", extras=not args.step_only)
        rec["breakdown_14b"] = breakdown_14b(w14, ms14, avg14, steps14)
        torch.cuda.empty_cache()
    if not args.no_cpu_baseline and args.only == "all":
        print("[bench] CPU oracle baseline", file=sys.stderr, flush=True)
        rec["cpu_baseline"] = cpu_baseline(w, heads=4 if args.workload == "14b" else None)
        if "breakdown_14b" in rec:
            rec["breakdown_14b"]["cpu_baseline"] = cpu_baseline(WORKLOADS["14b"], heads=4)
    print(json.dumps(rec), flush=True)


def breakdown_14b(w, ms_step, avg, steps):
    """The 14B-shaped step's parts with their roofline fractions (attention and
    Gram against the bf16 MFMA peak, the solve against the fp32 peak)."""
    f = flops(w)
    total = step_flops(w, f)

    def frac(fl, ms, peak):
        return round(fl / ms / 1e9 / peak, 4)

    sa = avg.get("solve_all_layers")
    return {
        "workload": w["name"], "heads": w["heads"], "head_dim": w["head_dim"], "chunk_queries": w["n_q"],
        "cache_len": w["cache_len"], "window": w["window"], "d": w["heads"] * w["head_dim"], "steps": steps,
        "ms_per_step": round(ms_step, 4), "tflops_step": round(total / (ms_step * 1e-3) / 1e12, 2),
        "attn_dual_ms": round(avg["attn_dual"], 4),
        "attn_dual_tflops": round(f["attn_dual"] / avg["attn_dual"] / 1e9, 1),
        "attn_dual_frac": frac(f["attn_dual"], avg["attn_dual"], PEAK_BF16_TFLOPS),
        "attn_local_ms": round(avg["attn_local"], 4),
        "attn_local_tflops": round(f["attn_local"] / avg["attn_local"] / 1e9, 1),
        "attn_local_frac": frac(f["attn_local"], avg["attn_local"], PEAK_BF16_TFLOPS),
        "accum_stats_ms": round(avg["accum_stats"], 4),
        "gram_tflops": round(f["gram"] / avg["accum_stats"] / 1e9, 1),
        "gram_frac": frac(f["gram"], avg["accum_stats"], PEAK_BF16_TFLOPS),
        "solve_ms": round(avg["solve"], 4),
        "solve_tflops": round(f["solve"] / avg["solve"] / 1e9, 2),
        "solve_frac_fp32_peak": frac(f["solve"], avg["solve"], PEAK_FP32_TFLOPS),
        "solve_all_layers": sa,
        "absorb": avg.get("absorb"),
        "dual_overhead": avg.get("dual_overhead"),
        "attn_zero_inputs": avg.get("attn_zero_inputs"),
        "per": "attention and accum_stats (discrepancy + Gram): ms per chunk call (4 per step); solve: ms per "
               "layer; fractions against 2500 TFLOP/s bf16 and 157.3 TFLOP/s fp32",
        "flop": f,
    }


if __name__ == "__main__":
    main()
