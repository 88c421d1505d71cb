"""Benchmark of the Thinker decoder layer on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-decode] [--no-cpu]

A step is one tri_layer_prefill call of the 7B-class dense layer over 8
sequences x 2048 tokens (hidden 3584, 28/4 heads, head_dim 128, SwiGLU 18944),
inputs seeded and already resident in HBM.  K timed steps are bracketed by
torch.cuda.synchronize() and HIP events on the launch stream; per-stage
durations come from the library's own HIP-event timers over the same timed
region.  The decode workload (batch 64, KV 4096, 32 steps) is timed as a
secondary result.  The full record (per-stage times, phase intensities,
secondary workloads) goes to stderr as one JSON line (and to --detail-out);
the last stdout line is a compact JSON summary of at most 4 KB.

Phases: for each workload (dense prefill, dense decode, MoE prefill, MoE
decode, mixed, the dense and MoE prefills with the per-head q/k RMSNorm
of the Qwen3-family attention block, and the dense prefill and decode with
the q/k/v bias of the Qwen2 family) the line carries the per-stage arithmetic intensity (the
library's work model: algorithmic flops over compulsory HBM bytes), the
phase's time-weighted intensity of Eq. 5 (weights: the stage times measured
in the profiled repetition), achieved TFLOP/s and GB/s per stage, and the
energy, shader clock, hotspot temperature and socket power over a >= 2 s loop.

Roofline: the dominant kernel of prefill is the fused gate/up + SwiGLU GEMM
(2 * 16384 * 37888 * 3584 flop per launch), priced against 2.5 PFLOP/s dense
bf16; decode's dominant kernel is split-KV attention, priced against 8 TB/s
on the K/V bytes it must read.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0
METRIC = "Thinker-layer prefill & decode tokens/s; % MFMA / HBM roofline; J/token"
TRAFFIC_SOURCE = ("profiles/traffic.txt: rocprofv3 FETCH_SIZE / WRITE_SIZE per launch, "
                  "copy-calibrated; null once the kernel source changed")


def linear_params(cfg) -> int:
    H, D = cfg.hidden, cfg.head_dim
    return H * cfg.qkv_rows + cfg.n_q_heads * D * H + 3 * cfg.ffn_dim * H


def prefill_flops(cfg, batch) -> float:
    pairs = sum((c + q) * (c + q + 1) // 2 - c * (c + 1) // 2 for c, q in zip(batch.ctx_len, batch.q_len))
    return 2.0 * linear_params(cfg) * batch.n_tokens + 4.0 * cfg.head_dim * cfg.n_q_heads * pairs


def profiled_traffic(kernel: str):
    """HBM bytes per launch of `kernel` from profiles/traffic.txt (rocprofv3
    FETCH_SIZE / WRITE_SIZE scaled by the copy calibration), or None when the
    kernel's source has changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic.txt")
    if not os.path.exists(path):
        return None
    for line in open(path):
        f = line.split()
        if len(f) < 2 or f[0] != "kernel" or f[1] != kernel:
            continue
        kv = dict(zip(f[2::2], f[3::2]))
        src = os.path.join(ROOT, kv["source"])
        if hashlib.sha256(open(src, "rb").read()).hexdigest() != kv["sha256"]:
            return None
        return (float(kv["fetch_kib"]) * 1024 * float(kv["fetch_factor"])
                + float(kv["write_kib"]) * 1024 * float(kv["write_factor"]))
    return None


class Energy:
    """Board energy counter of the GPU in use, read in-process through the
    amdsmi library (accumulator x resolution, microjoules); None when the
    library or the counter is unavailable."""

    def __init__(self):
        self.h = None
        try:
            import amdsmi
            import torch
            amdsmi.amdsmi_init()
            handles = amdsmi.amdsmi_get_processor_handles()
            h = handles[0] if len(handles) == 1 else None
            bus = getattr(torch.cuda.get_device_properties(0), "pci_bus_id", None)
            if h is None and bus is not None:
                for c in handles:
                    if int(str(amdsmi.amdsmi_get_gpu_device_bdf(c)).split(":")[1], 16) == bus:
                        h = c
            if h is not None:
                amdsmi.amdsmi_get_energy_count(h)
                self.amdsmi, self.h = amdsmi, h
        except Exception:
            self.h = None

    def joules(self):
        if self.h is None:
            return None
        try:
            e = self.amdsmi.amdsmi_get_energy_count(self.h)
            return e["energy_accumulator"] * e["counter_resolution"] * 1e-6
        except Exception:
            return None

    def sample(self):
        """Shader clock (MHz, mean over the XCDs that report one), hotspot
        temperature (C) and socket power (W) from the GPU metrics table."""
        if self.h is None:
            return None
        try:
            m = self.amdsmi.amdsmi_get_gpu_metrics_info(self.h)
        except Exception:
            return None

        def num(v):
            return float(v) if isinstance(v, (int, float)) and not isinstance(v, bool) else None

        clks = m.get("current_gfxclks")
        vals = [num(c) for c in clks] if isinstance(clks, (list, tuple)) else []
        vals = [v for v in vals if v is not None and v > 0]
        clk = sum(vals) / len(vals) if vals else (num(m.get("current_gfxclk"))
                                                 or num(m.get("average_gfxclk_frequency")))
        return {"gfxclk_mhz": clk, "hotspot_c": num(m.get("temperature_hotspot")),
                "socket_power_w": num(m.get("current_socket_power"))}


def _mean(samples, key):
    v = [x[key] for x in samples if x.get(key) is not None]
    return sum(v) / len(v) if v else None


def energy_loop(fn, min_s=2.0):
    """Joules per call of fn over a loop of at least min_s seconds (the counter
    updates every few ms), after one second at the same load, with average
    board power and the clock, temperature and power sampled while the GPU is
    busy; None without a counter."""
    import torch
    meter = Energy()
    if meter.h is None:
        return None
    # one second at the same load first: the metrics table (clock, socket
    # power) lags a change of load, so the samples reflect the steady state
    torch.cuda.synchronize()
    t_w = time.perf_counter()
    while time.perf_counter() - t_w < 1.0:
        for _ in range(4):
            fn()
        torch.cuda.synchronize()
    t0, j0, n = time.perf_counter(), meter.joules(), 0
    samples = []
    while True:
        fn()
        n += 1
        if n % 4 == 0:
            smp = meter.sample()  # work is still queued: a busy-GPU reading
            if smp:
                samples.append(smp)
            torch.cuda.synchronize()
            if time.perf_counter() - t0 >= min_s:
                break
    torch.cuda.synchronize()
    t1, j1 = time.perf_counter(), meter.joules()
    if j0 is None or j1 is None or j1 <= j0:
        return None
    return {"joules_per_call": (j1 - j0) / n, "avg_power_w": (j1 - j0) / (t1 - t0),
            "calls": n, "seconds": t1 - t0,
            "telemetry": {"gfxclk_mhz": _mean(samples, "gfxclk_mhz"),
                          "hotspot_c": _mean(samples, "hotspot_c"),
                          "socket_power_w": _mean(samples, "socket_power_w"),
                          "samples": len(samples)}}


def energy_json(energy, tokens_per_call):
    if energy is None:
        return None
    return {"joules_per_token": energy["joules_per_call"] / tokens_per_call,
            "avg_power_w": energy["avg_power_w"], "seconds": energy["seconds"],
            "source": "amdsmi board energy counter", "telemetry": energy["telemetry"]}


def prof_dict(p):
    return {p.name[i].decode(): {"launches": p.launches[i], "total_ms": p.total_ms[i]}
            for i in range(p.n_stages)}


def phase_report(tri, cfg, calls, decode, prof, reps, energy=None, tokens_per_call=None):
    """Per-stage arithmetic intensity (algorithmic flops / compulsory bytes, from
    the library's work model) and the phase's time-weighted intensity, Eq. 5,
    weighted by the stage times measured over `reps` repetitions of `calls`
    (a list of (q_len, ctx_len, expert_rows) host arrays)."""
    w = tri.work_sum([tri.layer_work(cfg, decode, q, c, er) for q, c, er in calls])
    ai = tri.phase_intensity(w, prof)
    stages = {}
    tot_f = tot_b = tot_ms = 0.0
    for i in range(w.n_stages):
        if not w.runs[i] or prof.total_ms[i] <= 0 or w.bytes[i] == 0:
            continue  # not launched, not timed, or a launch with no work
        ms = prof.total_ms[i]
        f, b = w.flops[i] * reps, w.bytes[i] * reps
        tot_f, tot_b, tot_ms = tot_f + f, tot_b + b, tot_ms + ms
        stages[w.name[i].decode()] = {
            "ms_per_call": ms / max(prof.launches[i], 1), "share": ms,
            "ai_flop_per_byte": w.flops[i] / w.bytes[i],
            "tflops": f / (ms / 1e3) / 1e12, "gbs": b / (ms / 1e3) / 1e9}
    for v in stages.values():
        v["share"] /= tot_ms
    out = {"ai_time_weighted": ai, "ai_aggregate": tot_f / tot_b,
           "tflops": tot_f / (tot_ms / 1e3) / 1e12, "gbs": tot_b / (tot_ms / 1e3) / 1e9,
           "stages": stages}
    if energy is not None:
        out["energy"] = energy_json(energy, tokens_per_call)
    return out


def cpu_baseline(wl, wb, kb, vb, xb, budget_s=12.0):
    """The CPU oracle (plain fp32 NumPy) on a bounded sample: whole sequences of
    the same workload, repeated until the time budget is used."""
    import oracle
    from synth import Batch, bf16_to_f32
    try:
        from threadpoolctl import threadpool_info
        threads = max((p.get("num_threads", 1) for p in threadpool_info()), default=os.cpu_count())
    except Exception:
        threads = os.cpu_count()
    w = {k: bf16_to_f32(v) for k, v in wb.items()}
    q = int(wl.batch.q_len[0])
    sub = Batch(wl.batch.slot[:1], wl.batch.ctx_len[:1], wl.batch.q_len[:1])
    x = bf16_to_f32(xb[:q])
    t0 = time.perf_counter()
    n_tok = 0
    reps = 0
    while True:
        oracle.layer_forward(wl.cfg, w, kb, vb, sub, x, dtype=np.float32)
        n_tok += q
        reps += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    dt = time.perf_counter() - t0
    return {"value": n_tok / dt, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{reps} x one {q}-token causal prefill sequence of the same layer "
                      f"(fp32 NumPy oracle), {dt:.1f} s"}


def run_prefill(args, tri, wl, wb, kb, vb, xb):
    import torch
    from paper_2606_29629_amd.workload import DeviceLayer, device_batch, device_cache, to_device_bf16
    dl = DeviceLayer(wl.cfg, wb)
    cache = device_cache(kb, vb)
    x = to_device_bf16(xb)
    db = device_batch(wl.batch)
    out = torch.empty_like(x)
    ws = torch.empty(tri.workspace_size(dl.cfg, db), dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        tri.layer_prefill(dl.cfg, dl.w, cache, db, x, out=out, workspace=ws)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def step():
        tri.layer_prefill(dl.cfg, dl.w, cache, db, x, out=out, workspace=ws)

    # Timed region: exactly `steps` layer calls, no per-stage events.
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = e0.elapsed_time(e1) / args.steps
    # Same steps again with the library's per-stage HIP events (kernel times).
    tri.profile_enable(True)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    praw = tri.profile_read(raw=True)
    tri.profile_enable(False)
    energy = energy_loop(step)
    phase = phase_report(tri, dl.cfg, [(wl.batch.q_len, wl.batch.ctx_len, None)], False, praw,
                         args.steps, energy, wl.batch.n_tokens)
    del dl, cache, x, out, ws
    torch.cuda.empty_cache()
    return ms, wall, prof_dict(praw), energy, phase


def run_decode(args, tri):
    import torch
    from paper_2606_29629_amd.workload import DeviceLayer, device_batch, device_cache, to_device_bf16
    from synth import make_cache, make_weights, make_x, workload
    wl = workload("dense_decode")
    wb = make_weights(wl.cfg, wl.seed)
    kb, vb = make_cache(wl.cfg, wl.n_slots, wl.max_seq, wl.seed)
    dl = DeviceLayer(wl.cfg, wb)
    cache = device_cache(kb, vb)
    del kb, vb
    steps = wl.decode_steps + 1
    batches, xs = [], []
    b = wl.batch
    for s in range(steps):
        batches.append(device_batch(b))
        xs.append(to_device_bf16(make_x(wl.cfg, b.n_tokens, wl.seed, step=s)))
        b = b.advanced()
    out = torch.empty_like(xs[0])
    ws_bytes = max(tri.workspace_size(dl.cfg, db) for db in batches)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    for s in range(min(steps, 4)):
        tri.layer_decode(dl.cfg, dl.w, cache, batches[s], xs[s], out=out, workspace=ws)
    torch.cuda.synchronize()
    reps = max(1, args.decode_reps)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def sweep():
        for s in range(steps):
            tri.layer_decode(dl.cfg, dl.w, cache, batches[s], xs[s], out=out, workspace=ws)

    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(reps):
        sweep()
    e1.record(stream)
    torch.cuda.synchronize()
    total_ms = e0.elapsed_time(e1)
    tri.profile_enable(True)
    for _ in range(reps):
        sweep()
    torch.cuda.synchronize()
    praw = tri.profile_read(raw=True)
    prof = prof_dict(praw)
    tri.profile_enable(False)
    energy = energy_loop(sweep)
    phase = phase_report(tri, dl.cfg, [(bb.host["q_len"], bb.host["ctx_len"], None)
                                       for bb in batches], True, praw, reps, energy,
                         steps * wl.batch.n_seqs)
    n_tok = reps * steps * wl.batch.n_seqs
    kv_bytes = sum(int(bb.host["ctx_len"].astype(np.int64).sum() + bb.n_seqs) for bb in batches) \
        * wl.cfg.n_kv_heads * wl.cfg.head_dim * 2 * 2
    act_bytes = steps * wl.batch.n_seqs * wl.cfg.n_q_heads * wl.cfg.head_dim * 2 * 2
    attn = prof["attn_decode"]
    attn_s = attn["total_ms"] / 1e3 / reps
    attn_gbs = (kv_bytes + act_bytes) / attn_s / 1e9
    step_bytes = (2 * linear_params(wl.cfg) + kv_bytes / steps)
    res = {
        "workload": "dense_decode: batch 64, KV 4096 -> 4127, 32 one-token steps",
        "tokens_per_s": n_tok / (total_ms / 1e3),
        "ms_per_step": total_ms / (reps * steps),
        "hbm_frac_step": step_bytes / (total_ms / 1e3 / (reps * steps)) / 1e9 / PEAK_HBM_GBS,
        "roofline": {"kernel": "attn_decode (split-KV partials; the LSE combine is a separate stage)",
                     "bound": "hbm",
                     "achieved": attn_gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": attn_gbs / PEAK_HBM_GBS, "traffic": profiled_traffic("attn_decode"),
                     "traffic_source": TRAFFIC_SOURCE},
        "stages_ms_per_step": {k: v["total_ms"] / (reps * steps) for k, v in prof.items() if v["launches"]},
    }
    if energy is not None:
        res["energy"] = energy_json(energy, steps * wl.batch.n_seqs)
    res["paged"] = paged_decode(tri, dl, cache, batches, xs, out, ws, reps, stream)
    del dl, cache, xs, out, ws
    torch.cuda.empty_cache()
    return res, phase


def paged_decode(tri, dl, cache, batches, xs, out, ws, reps, stream, block_size=64):
    """The same decode sweep on a paged copy of the cache (64-row blocks in a
    shuffled pool): step time and attention time."""
    import torch
    from paper_2606_29629_amd.workload import paged_from_contiguous
    k, v = cache
    pad = (-k.shape[2]) % block_size
    if pad:
        k = torch.nn.functional.pad(k, (0, 0, 0, pad))
        v = torch.nn.functional.pad(v, (0, 0, 0, pad))
    pc = paged_from_contiguous(k, v, block_size, seed=7, fill=0.0)
    del k, v
    steps = len(batches)

    def sweep():
        for s in range(steps):
            tri.layer_decode(dl.cfg, dl.w, pc, batches[s], xs[s], out=out, workspace=ws)

    sweep()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        sweep()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / (reps * steps)
    tri.profile_enable(True)
    sweep()
    torch.cuda.synchronize()
    prof = tri.profile_read()
    tri.profile_enable(False)
    res = {"block_size": block_size, "ms_per_step": ms,
           "tokens_per_s": batches[0].n_seqs / (ms / 1e3),
           "attn_decode_ms": prof["attn_decode"]["total_ms"] / steps}
    del pc
    torch.cuda.empty_cache()
    return res


def run_secondary(args, tri, name):
    """Time another workload (tokens/s and per-stage ms) for context."""
    import torch
    from paper_2606_29629_amd.workload import DeviceLayer, device_batch, device_cache, to_device_bf16
    from synth import make_cache, make_weights, make_x, workload
    wl = workload(name)
    wb = make_weights(wl.cfg, wl.seed)
    kb, vb = make_cache(wl.cfg, wl.n_slots, wl.max_seq, wl.seed)
    dl = DeviceLayer(wl.cfg, wb)
    cache = device_cache(kb, vb)
    del kb, vb, wb
    steps = wl.decode_steps + 1
    batches, xs = [], []
    b = wl.batch
    for s in range(steps):
        batches.append(device_batch(b))
        xs.append(to_device_bf16(make_x(wl.cfg, b.n_tokens, wl.seed, step=None if s == 0 and
                                        int(b.q_len.max()) > 1 else s)))
        b = b.advanced()
    decode = wl.batch.q_len.max() == 1
    fn = tri.layer_decode if decode else tri.layer_prefill
    out = torch.empty_like(xs[0])
    ws = torch.empty(max(tri.workspace_size(dl.cfg, db) for db in batches), dtype=torch.uint8,
                     device="cuda")
    for s in range(min(steps, 2)):
        fn(dl.cfg, dl.w, cache, batches[s], xs[s], out=out, workspace=ws)
    torch.cuda.synchronize()
    reps = 3
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def sweep(routes=None):
        for s in range(steps):
            r = None if routes is None else routes[s]
            fn(dl.cfg, dl.w, cache, batches[s], xs[s], out=out, workspace=ws, route_idx=r)

    e0.record(stream)
    for _ in range(reps):
        sweep()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / (reps * steps)
    tri.profile_enable(True)
    for _ in range(reps):
        sweep()
    torch.cuda.synchronize()
    praw = tri.profile_read(raw=True)
    tri.profile_enable(False)
    expert_rows = [None] * steps
    if getattr(wl.cfg, "n_experts", 0):
        routes = [torch.empty(db.n_tokens, wl.cfg.top_k, dtype=torch.int32, device="cuda")
                  for db in batches]
        sweep(routes)
        torch.cuda.synchronize()
        expert_rows = [np.bincount(r.cpu().numpy().ravel(), minlength=wl.cfg.n_experts)
                       for r in routes]
    energy = energy_loop(sweep)
    n_tok = wl.batch.n_tokens if not decode else wl.batch.n_seqs
    phase = phase_report(tri, dl.cfg, [(bb.host["q_len"], bb.host["ctx_len"], er)
                                       for bb, er in zip(batches, expert_rows)], bool(decode),
                         praw, reps, energy, n_tok * steps)
    res = {"workload": f"{name}: {wl.description}", "ms_per_step": ms,
           "tokens_per_s": n_tok / (ms / 1e3),
           "stages_ms_per_step": {k: v["total_ms"] / (reps * steps)
                                  for k, v in prof_dict(praw).items() if v["launches"]}}
    if expert_rows[0] is not None:
        loads = np.stack(expert_rows)
        res["expert_load"] = {"max_over_mean": float((loads.max(1) / loads.mean(1)).mean()),
                              "experts_touched": float((loads > 0).sum(1).mean())}
    if energy is not None:
        res["energy"] = energy_json(energy, n_tok * steps)
    del dl, cache, xs, out, ws
    torch.cuda.empty_cache()
    return res, phase


def fit_models(points, eta, ai_key):
    """Fits of the throughput models of Section III-C to sweep points: Eq. 1
    with eta the published peak flops per clock and beta the median of
    throughput / A.I. over the points whose Eq. 1 bound is the memory term,
    and Eq. 3 with omega (gamma = 0: the clock is not set, so its exponent
    cannot be separated) on the points past the ridge at their own clock.
    Adds each point's model predictions."""
    fit = {"eta_flop_per_clock": eta}
    have_f = [p for p in points if p.get("gfxclk_mhz")]
    if not have_f:
        return fit
    ratios = sorted(p["tflops"] * 1e12 / p[ai_key] for p in have_f
                    if p[ai_key] < 0.25 * eta * p["gfxclk_mhz"] * 1e6 / (PEAK_HBM_GBS * 1e9))
    beta = ratios[len(ratios) // 2] if ratios else None
    fit["eq1_beta_gbs"] = beta / 1e9 if beta else None
    num = den = 0.0
    for p in have_f:
        f = p["gfxclk_mhz"] * 1e6
        if p[ai_key] >= eta * f / (PEAK_HBM_GBS * 1e9):
            num += eta * f * p[ai_key] / (p["tflops"] * 1e12) - p[ai_key]
            den += 1
    fit["eq3_omega_flop_per_byte"] = num / den if den else None
    for p in have_f:
        f = p["gfxclk_mhz"] * 1e6
        a = p[ai_key]
        p["eq1_tflops"] = min(eta * f, (beta or 0) * a) / 1e12
        if fit["eq3_omega_flop_per_byte"] is not None:
            p["eq3_tflops"] = min(eta * f * a / (a + fit["eq3_omega_flop_per_byte"]),
                                  (beta or 0) * a) / 1e12
    return fit


def matmul_sweep(tri, eta):
    """The paper's roofline benchmark kernel (Section II-C, frequency-locked
    roofline benchmarking) without clock control: a matrix multiply C = A W^T
    through tri_linear, W [N, K] = [65536, 4096] (512 MiB, past the 256 MB
    Infinity Cache; K as in the layer's projections), swept over A.I. in
    {1, 25, 50, 100, 200} flop/B by the row count M (A.I. = M N K / (M K + N K
    + M N) for bf16 operands, so M = A.I. N K / (N K - A.I. (N + K))).  Per
    point: time per call, TFLOP/s, GB/s, and the shader clock and socket
    power over a 2 s loop after 1 s at the same load.  Synthetic normal
    operands."""
    import torch
    K, N = 4096, 65536
    g = torch.Generator(device="cuda").manual_seed(0)
    w = (torch.randn((N, K), device="cuda", generator=g) * 0.02).to(torch.bfloat16)
    out = []
    for ai_target in (1, 25, 50, 100, 200):
        M = max(1, round(ai_target * N * K / (N * K - ai_target * (N + K))))
        a = torch.randn((M, K), device="cuda", generator=g).to(torch.bfloat16)
        c = torch.empty((M, N), device="cuda", dtype=torch.bfloat16)
        need = tri.linear_workspace_size(M, N, K)
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device="cuda")
        call = lambda: tri.linear(a, w, out=c, workspace=ws)
        for _ in range(3):
            call()
        torch.cuda.synchronize()
        reps = 20
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            call()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        flops, byts = 2.0 * M * N * K, 2.0 * (M * K + N * K + M * N)
        en = energy_loop(call, min_s=2.0)
        tel = en["telemetry"] if en else {}
        pt = {"ai_target": ai_target, "rows": M, "ai": flops / byts, "ms_per_call": ms,
              "tflops": flops / (ms / 1e3) / 1e12, "gbs": byts / (ms / 1e3) / 1e9,
              "gfxclk_mhz": tel.get("gfxclk_mhz"), "socket_power_w": tel.get("socket_power_w"),
              "board_power_w": en["avg_power_w"] if en else None,
              "joules_per_tflop": en["joules_per_call"] / (flops / 1e12) if en else None}
        out.append(pt)
        print(json.dumps({"matmul_sweep_point": pt}), file=sys.stderr, flush=True)
        del a, c, ws
    del w
    torch.cuda.empty_cache()
    return out, fit_models(out, eta, "ai")


def ai_sweep(args, tri):
    """Arithmetic-intensity sweep under the GPU's own clock management (the
    paper's frequency-locked roofline, Section II-C, without clock control):
    the 7B dense layer at token counts from one decode token to a 16384-token
    prefill.  Per point: the layer's time-weighted A.I. (Eq. 5, from the work
    model and the measured stage times), achieved TFLOP/s and GB/s, and the
    shader clock and socket power over a 2 s loop after 1 s at the same load.  Then the throughput
    models are fitted to the points: Eq. 1 with eta the published peak flops
    per clock and beta fitted, and Eq. 3 with omega (gamma = 0: the clock is
    not set, so its exponent cannot be separated)."""
    import torch
    from paper_2606_29629_amd.workload import DeviceLayer, device_batch, device_cache, to_device_bf16
    from synth import Batch, layer_7b, make_cache, make_weights, make_x
    cfg = layer_7b()
    wb = make_weights(cfg, 0)
    dl = DeviceLayer(cfg, wb)
    points = []  # (label, decode, batch)
    for B in (1, 4, 16, 64, 128):
        points.append((f"decode B={B}, ctx 512", True,
                       Batch(np.arange(B, dtype=np.int32), np.full(B, 512, np.int32),
                             np.ones(B, np.int32))))
    for n, L in ((1, 256), (1, 1024), (2, 2048), (8, 2048)):
        points.append((f"prefill {n} x {L}", False,
                       Batch(np.arange(n, dtype=np.int32), np.zeros(n, np.int32),
                             np.full(n, L, np.int32))))
    eta = PEAK_BF16_TFLOPS * 1e12 / 2.4e9   # flops per clock (published peak at 2.4 GHz)
    out = []
    for label, decode, b in points:
        n_slots = b.n_seqs
        kb, vb = make_cache(cfg, n_slots, int((b.ctx_len + b.q_len).max()) + 64, 0)
        cache = device_cache(kb, vb)
        del kb, vb
        db = device_batch(b)
        x = to_device_bf16(make_x(cfg, b.n_tokens, 0, step=0 if decode else None))
        fn = tri.layer_decode if decode else tri.layer_prefill
        o = torch.empty_like(x)
        ws = torch.empty(tri.workspace_size(dl.cfg, db), dtype=torch.uint8, device="cuda")
        call = lambda: fn(dl.cfg, dl.w, cache, db, x, out=o, workspace=ws)
        for _ in range(3):
            call()
        torch.cuda.synchronize()
        reps = 20 if decode else 5
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            call()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        tri.profile_enable(True)
        for _ in range(reps):
            call()
        torch.cuda.synchronize()
        praw = tri.profile_read(raw=True)
        tri.profile_enable(False)
        w = tri.layer_work(dl.cfg, decode, b.q_len, b.ctx_len)
        ai = tri.phase_intensity(w, praw)
        flops = sum(w.flops[i] for i in range(w.n_stages))
        byts = sum(w.bytes[i] for i in range(w.n_stages))
        en = energy_loop(call, min_s=2.0)
        tel = en["telemetry"] if en else {}
        pt = {"point": label, "tokens": b.n_tokens, "ms_per_call": ms, "ai_time_weighted": ai,
              "ai_aggregate": flops / byts, "tflops": flops / (ms / 1e3) / 1e12,
              "gbs": byts / (ms / 1e3) / 1e9, "gfxclk_mhz": tel.get("gfxclk_mhz"),
              "socket_power_w": tel.get("socket_power_w"),
              "board_power_w": en["avg_power_w"] if en else None,
              "joules_per_token": en["joules_per_call"] / b.n_tokens if en else None}
        out.append(pt)
        print(json.dumps({"ai_sweep_point": pt}), file=sys.stderr, flush=True)
        del cache, db, x, o, ws
        torch.cuda.empty_cache()
    fit = fit_models(out, eta, "ai_time_weighted")
    mm, mm_fit = matmul_sweep(tri, eta)
    print(json.dumps({"ai_sweep": out, "fit": fit, "matmul_sweep": mm, "matmul_fit": mm_fit,
                      "ridge_flop_per_byte": PEAK_BF16_TFLOPS / PEAK_HBM_GBS * 1e3,
                      "layer": "7B dense (H 3584, 28/4 heads, D 128, F 18944), bf16"}))
    return 0


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--decode-reps", type=int, default=5)
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-secondary", action="store_true",
                    help="skip the MoE prefill / MoE decode / mixed-step context numbers")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device copy 3 times (HBM counter calibration)")
    ap.add_argument("--detail-out", default=None,
                    help="also write the full result record (phases, stages, secondary) here")
    ap.add_argument("--ai-sweep", action="store_true",
                    help="only run the arithmetic-intensity sweeps of the 7B layer and of the matrix-multiply kernel (clock, power, "
                         "Eq. 1 / Eq. 3 fits) and print it as one JSON line")
    args = ap.parse_args(argv)
    if args.gpus != 1:
        print(f"bench.py: this build runs on exactly one GPU (asked for {args.gpus}); "
              "the layer is not sharded across GPUs.", file=sys.stderr)
        return 2
    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.copy_calibration:
        n = 1 << 30
        src = torch.ones(n // 2, dtype=torch.bfloat16, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": n, "bytes_written": n, "launches": 3}))
        return 0
    import paper_2606_29629_amd as tri
    from synth import make_cache, make_weights, make_x, workload
    if args.ai_sweep:
        return ai_sweep(args, tri)

    wl = workload("dense_prefill")
    wb = make_weights(wl.cfg, wl.seed)
    kb, vb = make_cache(wl.cfg, wl.n_slots, wl.max_seq, wl.seed)
    xb = make_x(wl.cfg, wl.batch.n_tokens, wl.seed)
    ms, wall, prof, energy, prefill_phase = run_prefill(args, tri, wl, wb, kb, vb, xb)
    T = wl.batch.n_tokens
    flops = prefill_flops(wl.cfg, wl.batch)
    gu = prof["gate_up"]
    gu_ms = gu["total_ms"] / max(gu["launches"], 1)
    gu_flops = 2.0 * T * 2 * wl.cfg.ffn_dim * wl.cfg.hidden
    gu_tflops = gu_flops / (gu_ms / 1e3) / 1e12
    res = {
        "metric": METRIC,
        "value": T / (ms / 1e3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) activations, N(0,0.02) random-init weights)",
        "config": {"workload": "dense_prefill: 7B-class dense Thinker layer, 8 x 2048-token causal prefill",
                   "hidden": wl.cfg.hidden, "q_heads": wl.cfg.n_q_heads, "kv_heads": wl.cfg.n_kv_heads,
                   "head_dim": wl.cfg.head_dim, "ffn": wl.cfg.ffn_dim, "batch": 8, "seq_len": 2048,
                   "parallelism": "single GPU"},
        "layer_tflops": flops / (ms / 1e3) / 1e12,
        "layer_mfma_frac": flops / (ms / 1e3) / 1e12 / PEAK_BF16_TFLOPS,
        "roofline": {"kernel": "gate_up (fused SwiGLU GEMM)", "bound": "mfma", "achieved": gu_tflops,
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": gu_tflops / PEAK_BF16_TFLOPS,
                     "traffic": profiled_traffic("gate_up"),
                     "traffic_source": TRAFFIC_SOURCE,
                     "algorithmic_bytes": 2.0 * (T * wl.cfg.hidden + 2 * wl.cfg.ffn_dim * wl.cfg.hidden
                                                 + T * wl.cfg.ffn_dim)},
        "stages_ms_per_step": {k: v["total_ms"] / args.steps for k, v in prof.items() if v["launches"]},
        "wall_s_timed": wall,
    }
    if energy is not None:
        res["energy"] = energy_json(energy, T)
    # Time-weighted arithmetic intensity per phase (Eq. 5), per-stage A.I.,
    # energy, clock and temperature: the inputs of an A.I.-aware frequency policy.
    phases = {"ridge_flop_per_byte": PEAK_BF16_TFLOPS / PEAK_HBM_GBS * 1e3,
              "dense_prefill": prefill_phase}
    if not args.no_decode:
        res["decode"], phases["dense_decode"] = run_decode(args, tri)
    if not args.no_secondary:
        res["secondary"] = []
        for n in ("moe_prefill", "moe_decode", "mixed", "dense_prefill_qkn", "moe_prefill_qkn",
                  "dense_prefill_bias", "dense_decode_bias", "talker_prefill", "talker_decode"):
            r, phases[n] = run_secondary(args, tri, n)
            res["secondary"].append(r)
    res["phases"] = phases
    if not args.no_cpu:
        from synth import bf16_to_f32
        res["cpu_baseline"] = cpu_baseline(wl, wb, bf16_to_f32(kb), bf16_to_f32(vb), xb)
    # Full detail (phases, per-stage data, secondary workloads) to stderr and,
    # if asked, to a file; stdout ends with the compact summary line.
    detail = json.dumps(res)
    print(detail, file=sys.stderr, flush=True)
    if args.detail_out:
        with open(args.detail_out, "w") as f:
            f.write(detail + "\n")
    print(json.dumps(summary_line(res)))
    return 0


def _r(v, sig=4):
    """Round floats to `sig` significant digits (recursively) for the summary line."""
    if isinstance(v, float):
        return float(f"{v:.{sig}g}")
    if isinstance(v, dict):
        return {k: _r(x, sig) for k, x in v.items()}
    if isinstance(v, list):
        return [_r(x, sig) for x in v]
    return v


SUMMARY_MAX_BYTES = 4000


def summary_line(res):
    """The compact result line (<= 4 KB): the headline prefill metric with its
    roofline, the decode result with its roofline, energy per token, the
    secondary workloads' step times and the CPU baseline.  Per-stage data and
    the phase intensities stay in the detail record."""
    keys = ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
            "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
            "layer_tflops", "layer_mfma_frac", "roofline")
    out = {k: res[k] for k in keys if k in res}
    if res.get("energy"):
        e = res["energy"]
        out["energy"] = {"joules_per_token": e["joules_per_token"], "avg_power_w": e["avg_power_w"],
                         "gfxclk_mhz": e["telemetry"].get("gfxclk_mhz")}
    out["stages_ms_per_step"] = res.get("stages_ms_per_step")
    d = res.get("decode")
    if d:
        dd = {k: d[k] for k in ("workload", "ms_per_step", "tokens_per_s", "hbm_frac_step",
                                "roofline") if k in d}
        if d.get("energy"):
            dd["joules_per_token"] = d["energy"]["joules_per_token"]
        if d.get("paged"):
            dd["paged_ms_per_step"] = d["paged"]["ms_per_step"]
        out["decode"] = dd
    if res.get("secondary"):
        sec = {}
        for r in res["secondary"]:
            e = r.get("energy")
            sec[r["workload"].split(":")[0]] = {
                "ms_per_step": r["ms_per_step"], "tokens_per_s": r["tokens_per_s"],
                "joules_per_token": e["joules_per_token"] if e else None}
        out["secondary"] = sec
    if res.get("cpu_baseline"):
        out["cpu_baseline"] = res["cpu_baseline"]
    out = _r(out)
    # stay within the size the driver keeps, dropping the least important parts
    for drop in ("stages_ms_per_step", "secondary"):
        if len(json.dumps(out)) <= SUMMARY_MAX_BYTES:
            break
        out.pop(drop, None)
    return out


if __name__ == "__main__":
    sys.exit(main())
