#!/usr/bin/env python3
"""Benchmark of the mixed-precision MoE layer on one MI355X.

Default workload: one Mixtral-8x7B-shaped MoE layer (d_model 4096, d_ff
14336, 8 SwiGLU experts, top-2) decoding one token per step; experts 0-3
are cached fp16, experts 4-7 are cache misses served by their group-32 int4
copy when their gate is below 0.3 (Eq. 2 rule with T1 = 0.7 at top-2).

A step is one full pass of the layer (gate GEMV, top-k, Eq. 2 decision,
work list, expert up/down projections, combine) over one token.  Steps
cycle through R identical weight replicas at distinct addresses and 64
distinct token vectors, all resident in HBM before timing starts, so that
no step finds its expert weights in L2 or the Infinity Cache.

Prints one JSON line on stdout (progress goes to stderr):
  value          decode tokens/s (whole job, one GPU)
  roofline       dominant kernel (expert up-projection): algorithmic bytes
                 per launch / its mean duration from HIP events on the
                 launch stream, against the 8 TB/s HBM peak
  cpu_baseline   the float64 CPU oracle timed on the host cores on a
                 bounded sample of the same workload

Counter modes (run under rocprofv3 --pmc; they print one JSON line):
  --copy-calibration   a plain 256 MiB device copy, 5 launches, to scale the
                       FETCH_SIZE / WRITE_SIZE counters to bytes
  --pmc-pass           only the warmup + timed decode steps, with the mean
                       algorithmic up-projection bytes of those launches
The roofline "traffic" field is read from the committed counter summary
under profiles/ for the workload (decode_up_mixtral_t1_pmc.md for the
default) and is null when the kernel's source has changed since those
counters were taken.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.join(ROOT, "tests"))

METRIC = ("MoE-layer decode tokens/s + effective weight GB/s (% of HBM peak), 1 GPU")
HBM_PEAK_GBPS = 8000.0
MFMA_F16_PEAK_TFLOPS = 2500.0
N_STREAMS = 64
CSRC = os.path.join(ROOT, "paper_2411_01433_amd", "csrc")
# Counter summaries of each workload's dominant kernel (profiles/), and the
# source file that kernel is built from: the recorded traffic is used only
# while that source is unchanged.
PMC_SUMMARIES = {
    "mixtral_layer_decode_t1": ("decode_up_mixtral_t1_pmc.md", "decode.hip"),
    "mixtral_int8_layer_decode_t1": ("decode_up_mixtral_int8_t1_pmc.md", "decode.hip"),
    "mixtral_layer_decode_t8_skew": ("decode_up_mfma_mixtral_t8_skew_pmc.md", "decode_mfma.hip"),
    "phi_moe_stack32_decode_t4": ("decode_up_phi_stack32_t4_pmc.md", "decode.hip"),
    "mixtral_stack32_prefill_t512": ("prefill_up_mixtral_stack32_t512_pmc.md", "prefill.hip"),
}
# arithmetic type of the path: fp16 activations and dequantised weights into
# fp32 accumulation; the int8-model workload streams int8 / int2 copies
DTYPE = {"mixtral_int8_layer_decode_t1": "f16 (int8/int2 weights)"}


def source_sha256(workload):
    if workload not in PMC_SUMMARIES:
        return None
    src = os.path.join(CSRC, PMC_SUMMARIES[workload][1])
    with open(src, "rb") as fh:
        return hashlib.sha256(fh.read()).hexdigest()


def measured_traffic(workload):
    """HBM bytes per launch of the dominant kernel from the committed counter
    summary: FETCH_SIZE and WRITE_SIZE (KiB per dispatch), each scaled by
    what the counter reads for a copy of known size.  None when there is no
    summary for this workload or the kernel source changed."""
    if workload not in PMC_SUMMARIES:
        return None, "no counter summary for this workload"
    try:
        text = open(os.path.join(ROOT, "profiles", PMC_SUMMARIES[workload][0])).read()
    except OSError:
        return None, "no counter summary"
    m = re.search(r"<!-- traffic-json (\{.*?\}) -->", text, re.S)
    if not m:
        return None, "no traffic record in the counter summary"
    rec = json.loads(m.group(1))
    if rec.get("workload") != workload:
        return None, "counter summary is for another workload"
    if rec.get("source_sha256") != source_sha256(workload):
        return None, "kernel source changed since the counters were taken"
    b = (rec["fetch_kib_per_dispatch"] * rec["fetch_factor"]
         + rec["write_kib_per_dispatch"] * rec["write_factor"]) * 1024.0
    return b, "rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated"


def event_overhead_us(n=50, warm=10):
    """Cost of two HIP event records back to back after a kernel on the
    current stream (what an empty stage of the library's stage timing
    measures): the median of n pairs after `warm` untimed ones (single
    pairs occasionally read several times the typical value)."""
    import torch
    a = torch.zeros(256, device="cuda")
    pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
             for _ in range(warm + n)]
    for e0, e1 in pairs:
        a.add_(1.0)
        e0.record()
        e1.record()
    torch.cuda.synchronize()
    return float(np.median([e0.elapsed_time(e1) for e0, e1 in pairs[warm:]]) * 1e3)


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def matrix_bytes(rows, cols, bits):
    if bits == 16:
        return rows * cols * 2
    return rows * cols * bits // 8 + rows * (cols // 32) * 2


def expert_bytes(d, f, bits):
    return 2 * matrix_bytes(f, d, bits) + matrix_bytes(d, f, bits)


def copy_bits(tag, prec):
    """Bit width of the copy a (tag, precision class) pair streams: the high
    copy is fp16, or int8 for the int8-model tags (5, 6); the low copy is
    int4 for tags 1 and 3, else int2."""
    if prec == 0:
        return 8 if tag in (5, 6) else 16
    return 4 if tag in (1, 3) else 2


def decode_up_kernel_name(T, K, E):
    """The up-projection kernel the library runs for a decode step: the dot2
    kernel for 1-2 tokens, and up to 8 while T * K <= E; else the
    matrix-core kernel."""
    if T <= 2 or (T <= 8 and T * K <= E):
        return "decode_up_kernel"
    return "decode_up_mfma_kernel"


def step_bytes(wl, idx, prec, tags):
    """Algorithmic bytes of one step: every distinct (expert, precision) copy
    the step streams, plus the gate; and the up-projection's share."""
    d, f = wl.d_model, wl.d_ff
    copies = set()
    for e, p in zip(idx.ravel(), prec.ravel()):
        if p == 2:
            continue
        bits = copy_bits(int(tags[int(e)]), int(p))
        copies.add((int(e), bits))
    T, K = idx.shape
    n_pairs = int((prec != 2).sum())
    total = sum(expert_bytes(d, f, b) for _, b in copies) + wl.n_experts * d * 2
    up = (sum(2 * matrix_bytes(f, d, b) for _, b in copies)
          + T * d * 2 + n_pairs * f * 2)
    return total, up


def down_bytes(wl, idx, prec, tags):
    """Algorithmic bytes of one down-projection launch: the W2 part of every
    distinct copy, the h rows read (fp16) and the expert outputs written
    (fp32), one per routed (token, slot) pair."""
    d, f = wl.d_model, wl.d_ff
    copies = {(int(e), copy_bits(int(tags[int(e)]), int(p)))
              for e, p in zip(idx.ravel(), prec.ravel()) if p != 2}
    n_pairs = int((prec != 2).sum())
    return sum(matrix_bytes(d, f, b) for _, b in copies) + n_pairs * f * 2 + n_pairs * d * 4


def cpu_info():
    info = {"cpus_affinity": len(os.sched_getaffinity(0)), "nproc": os.cpu_count()}
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                info["model"] = ln.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return info


def blas_threads():
    try:
        from threadpoolctl import threadpool_info
        n = [p.get("num_threads", 0) for p in threadpool_info()
             if p.get("user_api") == "blas"]
        return max(n) if n else 1
    except Exception:
        return 1


def run_decode_layer(args):
    import torch
    import gpu_support as S
    import paper_2411_01433_amd as P
    from synth import configs as C

    wl = C.BY_NAME[args.workload]
    assert wl.n_layers == 1 and wl.mode == "decode"
    dev = torch.device("cuda:0")
    T, K, d = wl.n_tokens, wl.top_k, wl.d_model
    tags = C.layer_tags(wl, 0)
    R = args.replicas
    log(f"workload {wl.name}: generating {R} weight replicas in HBM")
    layers, keep = [], []
    for r in range(R):
        w = S.device_layer_weights(wl, 0, device=dev)
        keep.append(w)
        layers.append(S.make_layer(wl, tags, w, max_tokens=T))
    xs = torch.from_numpy(np.stack([C.hidden_states(wl, stream=s) for s in range(N_STREAMS)])).to(dev)
    n_all = args.warmup + args.steps
    y = torch.empty((N_STREAMS, T, d), dtype=torch.float32, device=dev)
    idx = torch.empty((n_all, T, K), dtype=torch.int32, device=dev)
    gw = torch.empty((n_all, T, K), dtype=torch.float32, device=dev)
    prec = torch.empty((n_all, T, K), dtype=torch.int8, device=dev)
    torch.cuda.synchronize()

    def step(i, r=None):
        s = i % N_STREAMS
        L = layers[(i % R) if r is None else r]
        L.decode_step(xs[s], y[s], idx[i], gw[i], prec[i])

    log("warmup", args.warmup)
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    log("timing", args.steps, "steps")
    ev0.record()
    for i in range(args.warmup, n_all):
        step(i)
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / args.steps

    idx_h, prec_h = idx.cpu().numpy(), prec.cpu().numpy()
    if args.pmc_pass:
        ups = [step_bytes(wl, idx_h[i], prec_h[i], tags)[1] for i in range(n_all)]
        return {"mode": "pmc-pass", "workload": wl.name, "launches": n_all,
                "up_bytes_per_launch_mean": float(np.mean(ups)),
                "source_sha256": source_sha256(wl.name)}, None
    per = [step_bytes(wl, idx_h[i], prec_h[i], tags) for i in range(args.warmup, n_all)]
    b_total = float(np.mean([p[0] for p in per]))
    b_up = float(np.mean([p[1] for p in per]))

    # hot number: one replica, same token (weights may sit in the MALL)
    hot_steps = max(20, args.steps // 4)
    for i in range(5):
        layers[0].decode_step(xs[0], y[0], idx[0], gw[0], prec[0])
    torch.cuda.synchronize()
    ev0.record()
    for i in range(hot_steps):
        layers[0].decode_step(xs[0], y[0], idx[0], gw[0], prec[0])
    ev1.record()
    torch.cuda.synchronize()
    ms_hot = ev0.elapsed_time(ev1) / hot_steps

    # per-step distribution: one event between consecutive steps
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    evs[0].record()
    for j, i in enumerate(range(args.warmup, n_all)):
        step(i)
        evs[j + 1].record()
    torch.cuda.synchronize()
    per_step = np.array([evs[j].elapsed_time(evs[j + 1]) * 1e3 for j in range(args.steps)])
    q10, q50, q90 = (float(v) for v in np.percentile(per_step, [10, 50, 90]))

    # stage-timed pass (events between kernels on the launch stream)
    log("stage timing pass")
    for L in layers:
        L.enable_timing(True)
    for i in range(args.warmup, n_all):
        step(i)
    torch.cuda.synchronize()
    tot = np.zeros(4)
    calls = 0
    for L in layers:
        t, n = L.stage_times()
        tot += np.array(t)
        calls += n
        L.enable_timing(False)
    stage_us = (tot / max(calls, 1) * 1e3).tolist()
    # Stage 3 (the residual RMSNorm) launches nothing in a plain decode step,
    # so its event pair measures the pure cost of the event records between
    # two kernels on this stream; it is subtracted from the up stage.
    event_us = stage_us[3]
    up_us = stage_us[1] - event_us
    achieved = b_up / (up_us * 1e-6) / 1e9
    traffic, traffic_note = measured_traffic(wl.name)

    out = {
        "metric": METRIC,
        "value": T / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": DTYPE.get(wl.name, "f16"), "data": "synthetic",
        "config": {"workload": wl.name, "d_model": d, "d_ff": wl.d_ff,
                   "n_experts": wl.n_experts, "top_k": K, "tokens_per_step": T,
                   "layers": 1, "weight_replicas": R, "token_streams": N_STREAMS,
                   "tags": wl.note},
        "effective_weight_GBps": b_total / (ms * 1e-3) / 1e9,
        "pct_hbm_peak": 100.0 * b_total / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
        "bytes_per_step": b_total,
        "hot_tokens_per_s": T / (ms_hot * 1e-3),
        "step_us_p10_p50_p90": [q10, q50, q90],
        "stage_us": dict(zip(["route", "up", "down_combine", "empty"], stage_us)),
        "event_overhead_us": event_us,
        "roofline": {"bound": "hbm",
                     "kernel": decode_up_kernel_name(T, wl.top_k, wl.n_experts),
                     "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS, "traffic": traffic,
                     "traffic_source": traffic_note,
                     "bytes_per_launch": b_up, "mean_launch_us": up_us,
                     "timing": "HIP events between kernels on the launch stream, "
                               "minus the same run's empty-stage event overhead"},
    }
    return out, (wl, tags, xs, y, idx, gw, prec, layers)


def stack_bytes_flops(wl, idx, prec, tags_per_layer):
    """Algorithmic bytes (distinct expert copies + gates) and FLOPs of one pass
    over the stack, from the routing each layer chose."""
    d, f = wl.d_model, wl.d_ff
    b = fl = 0
    for l in range(wl.n_layers):
        b += step_bytes(wl, idx[l], prec[l], tags_per_layer[l])[0]
        fl += int((prec[l] != 2).sum()) * 2 * 3 * d * f
    return b, fl


def run_stack(args):
    """32-layer stacks (residual glue between layers): the Phi-MoE-shaped
    decode stack (4 tokens) or the Mixtral-shaped prefill stack (512).  A
    step is one pass of the whole stack."""
    import torch
    import gpu_support as S
    import paper_2411_01433_amd as P
    from synth import configs as C

    wl = C.BY_NAME[args.workload]
    dev = torch.device("cuda:0")
    T, K, d, NL = wl.n_tokens, wl.top_k, wl.d_model, wl.n_layers
    log(f"workload {wl.name}: generating {NL} layers in HBM")
    layers, keep, tags_l = [], [], []
    for l in range(NL):
        tags = C.layer_tags(wl, l)
        w = S.device_layer_weights(wl, l, device=dev)
        keep.append(w)
        tags_l.append(tags)
        layers.append(S.make_layer(wl, tags, w, max_tokens=T))
        if l > 0:  # the layers run in turn: one workspace serves them all
            layers[l].share_workspace(layers[0])
    h0 = torch.from_numpy(C.hidden_states(wl).astype(np.float32)).to(dev)
    h = torch.empty_like(h0)
    # the first layer's input, by the library's own RMSNorm of the glue
    x_first = torch.empty((T, d), dtype=torch.float16, device=dev)
    P.rmsnorm(h0, x_first)
    xb = [torch.empty_like(x_first), torch.empty_like(x_first)]
    idx = torch.empty((NL, T, K), dtype=torch.int32, device=dev)
    gw = torch.empty((NL, T, K), dtype=torch.float32, device=dev)
    prec = torch.empty((NL, T, K), dtype=torch.int8, device=dev)
    prefill = wl.mode == "prefill"

    # decode stacks take the residual stream itself (moe_decode_step_prenorm:
    # each layer forms its own input norm inside its router); --glue residual
    # runs the separate norm kernel after every layer instead
    prenorm = not prefill and args.glue == "prenorm"

    def step():
        h.copy_(h0)
        xb[0].copy_(x_first)
        for l, L in enumerate(layers):
            xi, xo = xb[l % 2], xb[(l + 1) % 2]
            if prefill:
                L.prefill_residual(xi, h, xo, idx[l], gw[l], prec[l])
            elif prenorm:
                L.decode_step_prenorm(h, xi, idx[l], gw[l], prec[l])
            else:
                L.decode_step_residual(xi, h, xo, idx[l], gw[l], prec[l])

    # --graph: one pass of the stack (the two input copies and every
    # layer's kernels) captured once in a HIP graph and replayed per step.
    # Measured slower than launching from the host (Phi stack 4.77 -> 4.93
    # ms per pass, prefill stack unchanged): the device is not waiting for
    # launches, so eager launch is the default.
    graph = None
    if args.graph and not args.pmc_pass:
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()  # untimed pass before capture
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        torch.cuda.synchronize()

    def run():
        if graph is not None:
            graph.replay()
        else:
            step()

    log("warmup", args.warmup)
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    log("timing", args.steps, "steps", "(graph replays)" if graph is not None else "(eager)")
    ev0.record()
    for _ in range(args.steps):
        run()
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / args.steps
    idx_h, prec_h = idx.cpu().numpy(), prec.cpu().numpy()
    ups = [step_bytes(wl, idx_h[l], prec_h[l], tags_l[l])[1] for l in range(NL)]
    if args.pmc_pass:
        downs = [down_bytes(wl, idx_h[l], prec_h[l], tags_l[l]) for l in range(NL)]
        return {"mode": "pmc-pass", "workload": wl.name,
                "launches": NL * (args.warmup + args.steps),
                "up_bytes_per_launch_mean": float(np.mean(ups)),
                "down_bytes_per_launch_mean": float(np.mean(downs)),
                "source_sha256": source_sha256(wl.name)}, None
    b, fl = stack_bytes_flops(wl, idx_h, prec_h, tags_l)
    up_flops = [int((prec_h[l] != 2).sum()) * 2 * 2 * d * wl.d_ff for l in range(NL)]

    # per-pass distribution: one event between consecutive passes
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    evs[0].record()
    for j in range(args.steps):
        run()
        evs[j + 1].record()
    torch.cuda.synchronize()
    per_pass = np.array([evs[j].elapsed_time(evs[j + 1]) for j in range(args.steps)])
    p10, p50, p90 = (float(v) for v in np.percentile(per_pass, [10, 50, 90]))

    log("stage timing pass")
    for L in layers:
        L.enable_timing(True)
    for _ in range(max(2, args.steps // 2)):
        step()
    torch.cuda.synchronize()
    tot = np.zeros(4)
    calls = 0
    for L in layers:
        t, n = L.stage_times()
        tot += np.array(t)
        calls += n
        L.enable_timing(False)
    stage_us = (tot / max(calls, 1) * 1e3).tolist()
    ev_us = event_overhead_us()
    up_us = stage_us[1] - ev_us
    up_b, up_fl = float(np.mean(ups)), float(np.mean(up_flops))
    achieved = up_b / (up_us * 1e-6) / 1e9
    mfma_achieved = up_fl / (up_us * 1e-6) / 1e12
    traffic, traffic_note = measured_traffic(wl.name)
    t_s = ms * 1e-3
    frac = max(b / 8e12, fl / 2.5e15) / t_s
    kernel = "prefill_up_kernel" if prefill else (
        decode_up_kernel_name(T, K, wl.n_experts))
    out = {
        "metric": METRIC, "value": T / t_s, "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": DTYPE.get(wl.name, "f16"), "data": "synthetic",
        "config": {"workload": wl.name, "d_model": d, "d_ff": wl.d_ff,
                   "n_experts": wl.n_experts, "top_k": K, "tokens_per_step": T,
                   "layers": NL, "mode": wl.mode, "tags": wl.note,
                   "launch": "hipGraph replay of the whole pass" if graph is not None else "eager",
                   "glue": "prefill residual" if prefill else args.glue},
        "effective_weight_GBps": b / t_s / 1e9,
        "pct_hbm_peak": 100.0 * b / t_s / 1e9 / HBM_PEAK_GBPS,
        "bytes_per_step": b, "flops_per_step": fl,
        "mfma_util_step": fl / t_s / 2.5e15 if prefill else None,
        "roofline_step": {"bound": "hbm" if b / 8e12 >= fl / 2.5e15 else "mfma",
                          "frac": frac},
        "pass_ms_p10_p50_p90": [p10, p50, p90],
        "stage_us_per_layer": dict(zip(["route", "up", "down", "glue"], stage_us)),
        "event_overhead_us": ev_us,
        "roofline": {"bound": "hbm", "kernel": kernel,
                     "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS, "traffic": traffic,
                     "traffic_source": traffic_note,
                     "bytes_per_launch": up_b, "mean_launch_us": up_us,
                     "flops_per_launch": up_fl,
                     "mfma_achieved_TFLOPs": mfma_achieved,
                     "mfma_frac": mfma_achieved / MFMA_F16_PEAK_TFLOPS,
                     "timing": "HIP events between kernels on the launch stream, "
                               "minus the event-record overhead measured in the same run"},
    }
    return out, (wl, tags_l, layers, x_first, h0, idx, gw, prec)


def stack_cpu_baseline(args, state, out):
    """The oracle streamed one layer at a time on a bounded sample: layer 0
    of the stack, its first n tokens (the device's own layer input), with
    the expert copies prepared beforehand (excluded and reported).  Passes
    over the sample repeat until the time budget is spent; the stack rate
    is tokens per second through all n_layers layers at that per-layer
    cost."""
    import torch
    import gpu_support as S
    from oracle import moe_oracle as O
    from synth import configs as C

    wl, tags_l, layers, x_first, h0, idx, gw, prec = state
    NL = wl.n_layers
    n = min(args.cpu_tokens if wl.mode == "prefill" else wl.n_tokens, wl.n_tokens)
    x_h = x_first.cpu().numpy()[:n]
    h_h = h0.cpu().numpy()[:n].astype(np.float64)
    tags = tags_l[0]
    wg16 = C.router_weight(wl, 0)
    experts = S.HostExperts(wl, 0, tags)
    log(f"oracle: preparing the experts layer 0 uses for {n} tokens")
    t0 = time.perf_counter()
    r0 = O.route(x_h, wg16, tags, wl.top_k, wl.t1, wl.t2)
    for t in range(n):
        for k in range(wl.top_k):
            if r0.prec[t, k] != O.PREC_SKIP:
                experts[int(r0.idx[t, k])].weights(int(r0.prec[t, k]))
    prep_s = time.perf_counter() - t0
    log(f"oracle: timing (budget {args.cpu_seconds}s)")
    t0 = time.perf_counter()
    done = passes = 0
    while True:
        r = O.route(x_h, wg16, tags, wl.top_k, wl.t1, wl.t2)
        y = O.layer_output(x_h, experts, r)
        O.residual_step(h_h, y, O.RMS_EPS)
        done += n
        passes += 1
        if time.perf_counter() - t0 > args.cpu_seconds:
            break
    dt = time.perf_counter() - t0
    out["cpu_baseline"] = {
        "value": done / dt / NL, "unit": "tokens/s", "cores": blas_threads(),
        "kind": "oracle",
        "sample": (f"layer 0 of the {NL}-layer stack, its first {n} tokens (gate, top-k, "
                   f"Eq. 2, experts, residual glue), {passes} passes ({done} token-layers, "
                   f"{dt:.1f}s); rate scaled to all {NL} layers; float64 numpy oracle with the "
                   f"expert copies already prepared ({prep_s:.1f}s, excluded)"),
        "seconds": dt, "host": cpu_info()}


def run_predictor(args):
    """Stacking Computer timing (Section 3.3, the comparison of Fig. 17a):
    one stacked launch over the gates of p = 1..8 layers ahead against the
    sequential way, p one-layer predictions launched one after the other.
    One decode token; Mixtral-shaped (8 experts) and Phi-MoE-shaped (16)
    gates.  The gates are small (64-128 KiB per layer) and stay in L2."""
    import torch
    import paper_2411_01433_amd as P
    from synth import configs as C

    res = {}
    for wl in (C.MIXTRAL_PREFILL, C.PHI_STACK):
        d, E, K, T = wl.d_model, wl.n_experts, wl.top_k, 1
        gates = [torch.from_numpy(C.router_weight(wl, l)).cuda() for l in range(1, 9)]
        x = torch.from_numpy(C.hidden_states(wl)[:T]).cuda()
        stacked = {p: P.MoePredictor(d, E, K, T, gates[:p]) for p in range(1, 9)}
        single = [P.MoePredictor(d, E, K, T, [g]) for g in gates]
        cd = torch.zeros((8,), dtype=torch.int64, device="cuda")
        fm = torch.empty((1,), dtype=torch.int32, device="cuda")
        pre = torch.empty((1,), dtype=torch.int64, device="cuda")

        def timed(fn, n):
            for _ in range(10):
                fn()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(n):
                fn()
            e1.record()
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) / n * 1e3

        row = {}
        for p in range(1, 9):
            ip = torch.empty((T, p, K), dtype=torch.int32, device="cuda")
            i1 = torch.empty((T, 1, K), dtype=torch.int32, device="cuda")
            t_st = timed(lambda: stacked[p].predict(x, cd[:p], ip, fm, pre), args.steps)
            t_seq = timed(lambda: [single[j].predict(x, cd[:1], i1, fm, pre)
                                   for j in range(p)], args.steps)
            row[p] = {"stacked_us": t_st, "sequential_us": t_seq}
            log(f"{wl.name} p={p}: stacked {t_st:.2f} us, sequential {t_seq:.2f} us")
        res[f"E{E}_d{d}"] = row
        for pr in list(stacked.values()) + single:
            pr.destroy()
    return {"metric": "Stacking Computer: time per prediction vs layers ahead p",
            "unit": "us", "tokens": 1, "steps": args.steps, "data": "synthetic",
            "note": "stacked = one launch over the p stacked gates; sequential = p "
                    "one-layer launches back to back on the stream",
            "results": res}


def run_cache(args):
    """Mixed-precision expert cache manager (Section 3.4): miss penalty of
    each replacement policy on a seeded Mixtral-shaped synthetic trace, the
    Eq. 3 weights chosen on a separate calibration trace (grid of step 1/4
    over the simplex), and the manager's replay rate against the oracle.
    Host-side mode: no GPU work."""
    import itertools
    import numpy as np
    import paper_2411_01433_amd as P
    from synth import traces as TR
    L, E, K = 32, 8, 2
    hi_cap, lo_cap = L * E // 4, L * E // 8
    seqs, seq_len = 8, 128
    cal = TR.expert_trace(7, seqs, seq_len, L, E, K)
    test = TR.expert_trace(8, seqs, seq_len, L, E, K)
    n_tok = seqs * seq_len

    def penalty(w, tr):
        c = P.MoeCache(L, E, hi_cap, lo_cap, *w, bits_hi=16, bits_lo=4, miss_cost=1.0)
        c.replay(*tr)
        pen, hm, lm, hits = c.stats()
        c.destroy()
        return pen, hm, lm, hits

    grid = [w for w in itertools.product(range(5), repeat=4) if sum(w) == 4]
    grid = [tuple(v / 4 for v in w) for w in grid]
    best = min(grid, key=lambda w: (penalty(w, cal)[0], w))
    res = {}
    for name, w in (("lru", (1, 0, 0, 0)), ("lfu", (0, 1, 0, 0)), ("lhu", (0, 0, 1, 0)),
                    ("fld", (0, 0, 0, 1)), ("equal", (0.25,) * 4), ("calibrated", best)):
        pen, hm, lm, hits = penalty(w, test)
        res[name] = {"weights": list(w), "penalty_per_token": pen / n_tok,
                     "hi_misses": hm, "lo_misses": lm, "hits": hits}
        log(f"{name:10s} w={w} penalty/token {pen / n_tok:.4f} "
            f"hi-miss {hm} lo-miss {lm} hits {hits}")
    # replay rate of the library and of the oracle (the oracle on a sample)
    c = P.MoeCache(L, E, hi_cap, lo_cap, *best, bits_hi=16, bits_lo=4)
    t0 = time.perf_counter()
    reps = 20
    for _ in range(reps):
        c.replay(*test)
    lib_s = (time.perf_counter() - t0) / reps
    c.destroy()
    n_uses = len(test[0])
    out = {"metric": "expert-cache miss penalty per token (C units) and manager uses/s",
           "unit": "uses/s", "value": n_uses / lib_s, "higher_is_better": True,
           "data": "synthetic", "dtype": "f64",
           "config": {"workload": "mixtral_shaped_cache_trace", "n_layers": L, "n_experts": E,
                      "top_k": K, "hi_capacity": hi_cap, "lo_capacity": lo_cap,
                      "sequences": seqs, "tokens_per_sequence": seq_len, "uses": n_uses,
                      "bits_hi": 16, "bits_lo": 4},
           "policies": res, "us_per_token": lib_s / n_tok * 1e6}
    if not args.no_cpu_baseline:
        from oracle import cache_oracle as CO
        cfg = CO.CacheConfig(L, E, hi_cap, lo_cap, *best, bits_hi=16, bits_lo=4)
        m = min(n_uses, 20000)
        sample = [tuple(int(a[i]) for a in test[:4]) for i in range(m)]
        t0 = time.perf_counter()
        CO.replay(cfg, sample, sequence_starts=[0])
        dt = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": m / dt, "unit": "uses/s", "cores": 1, "kind": "oracle",
                               "sample": f"first {m} uses of the same trace, Python oracle",
                               "seconds": dt}
    return out


def run_loading(args):
    """Dynamic Expert Loader on MI355X (Section 3.2, Fig. 6; Section 2.2:
    expert loading dominates offloaded inference): one Mixtral-shaped expert loaded from pinned host
    storage into device slots at fp16, int4 and int2 on a copy stream (HIP
    events on that stream), and the 1-token decode step of a resident
    Mixtral-shaped layer timed alone and while loads run beside it."""
    import numpy as np
    import torch
    import paper_2411_01433_amd as P
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import gpu_support as S
    from synth import configs as C
    wl = C.MIXTRAL_T1
    d, f = wl.d_model, wl.d_ff
    weights = S.device_layer_weights(wl, 0)
    wg, w1, w3, w2 = weights
    side = torch.cuda.Stream()
    res = {}
    reps = max(3, min(args.steps, 10))
    for bits in (4, 2):
        st = P.MoeStore(d, f, 1, bits)
        st.put(0, w1[0], w3[0], w2[0])
        for high in ((True, False) if bits == 4 else (False,)):
            dst = st.slots(high)
            nbytes = 3 * (st.fp16_bytes if high else st.code_bytes + st.scale_bytes)
            st.load(0, high, dst, stream=side)
            side.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(side)
            for _ in range(reps):
                st.load(0, high, dst, stream=side)
            e1.record(side)
            side.synchronize()
            ms = e0.elapsed_time(e1) / reps
            name = "fp16" if high else f"int{bits}"
            res[name] = {"bytes": nbytes, "ms_per_expert": ms, "GBps": nbytes / ms / 1e6}
            log(f"load {name}: {nbytes / 1e6:.1f} MB in {ms:.2f} ms -> {nbytes / ms / 1e6:.1f} GB/s")
            del dst
        st.destroy()
    # decode alone vs with loads beside it
    L = S.make_layer(wl, C.layer_tags(wl, 0), weights, max_tokens=1)
    x = torch.from_numpy(C.hidden_states(wl)).cuda()
    y = torch.empty((1, d), device="cuda")
    st = P.MoeStore(d, f, 1, 4)
    st.put(0, w1[1], w3[1], w2[1])
    dst = st.slots(True)

    def decode_ms(n, with_loads):
        for _ in range(5):
            L.decode_step(x, y)
        torch.cuda.synchronize()
        if with_loads:
            for _ in range(max(1, n // 40)):
                st.load(0, True, dst, stream=side)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(n):
            L.decode_step(x, y)
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / n

    alone = decode_ms(200, False)
    beside = decode_ms(200, True)
    torch.cuda.synchronize()
    L.destroy()
    st.destroy()
    ratio = res["fp16"]["ms_per_expert"] / res["int4"]["ms_per_expert"]
    log(f"fp16 / int4 load time {ratio:.2f}x (bytes ratio 16 : 4.5 = 3.56); decode step "
        f"{alone * 1e3:.1f} us alone, {beside * 1e3:.1f} us beside loads")
    return {"metric": "expert load time host->HBM per Mixtral-shaped expert, by precision",
            "unit": "ms", "higher_is_better": False, "data": "synthetic", "dtype": "f16",
            "config": {"workload": "mixtral_expert_load", "d_model": d, "d_ff": f,
                       "storage": "hipHostMalloc pinned host memory", "reps": reps},
            "loads": res, "fp16_over_int4": ratio,
            "decode_step_us": {"alone": alone * 1e3, "beside_loads": beside * 1e3},
            "note": "the paper's loading bottleneck (Section 2.2) measured over the MI355X "
                    "host link; the hot path itself keeps every copy in HBM"}


def parity_and_cpu(args, state, out):
    """Check sampled steps against the oracle and time the oracle itself."""
    import torch
    import gpu_support as S
    from oracle import moe_oracle as O
    from synth import configs as C

    wl, tags, xs, y, idx, gw, prec, layers = state
    T, d = wl.n_tokens, wl.d_model
    n_sample = min(args.cpu_tokens, N_STREAMS)
    # device results for the sample, fresh, on replica 0
    ys = []
    for s in range(n_sample):
        layers[0].decode_step(xs[s], y[s], idx[s], gw[s], prec[s])
    torch.cuda.synchronize()
    y_h, idx_h, w_h, prec_h = (y.cpu().numpy(), idx.cpu().numpy(), gw.cpu().numpy(),
                              prec.cpu().numpy())
    x_h = xs.cpu().numpy()
    wg16 = C.router_weight(wl, 0)
    experts = S.HostExperts(wl, 0, tags)
    log(f"oracle: preparing experts for {n_sample} sample steps")
    t0 = time.perf_counter()
    routes = []
    for s in range(n_sample):
        r, _ = S.check_routing(x_h[s], wg16, tags, wl.top_k, wl.t1, wl.t2,
                               idx_h[s], w_h[s], prec_h[s])
        routes.append(r)
        for t in range(T):
            for k in range(wl.top_k):
                if r.prec[t, k] != O.PREC_SKIP:
                    experts[int(r.idx[t, k])].weights(int(r.prec[t, k]))
    prep_s = time.perf_counter() - t0
    log(f"oracle: timing (budget {args.cpu_seconds}s)")
    # the sampled steps are checked once and passed over again until the
    # time budget is spent (a bounded sample of CPU work)
    errs = []
    t0 = time.perf_counter()
    done = passes = 0
    while True:
        for s in range(n_sample):
            r = O.route(x_h[s], wg16, tags, wl.top_k, wl.t1, wl.t2,
                        forced_idx=routes[s].idx)
            r.prec = routes[s].prec
            y_ref = O.layer_output(x_h[s], experts, r)
            done += 1
            if passes == 0:
                errs.append(float(S.normwise(y_h[s], y_ref).max()))
        passes += 1
        if time.perf_counter() - t0 > args.cpu_seconds:
            break
    dt = time.perf_counter() - t0
    out["parity"] = {"steps_checked": len(errs), "max_normwise_err": max(errs),
                     "tol": S.TOL, "ok": max(errs) <= S.TOL}
    out["cpu_baseline"] = {
        "value": done * T / dt, "unit": "tokens/s", "cores": blas_threads(),
        "kind": "oracle",
        "sample": (f"{n_sample} decode steps (token streams 0..{n_sample - 1}) of the "
                   f"same layer, {passes} passes ({done} steps, {dt:.1f}s); float64 "
                   f"numpy oracle with the expert copies already prepared "
                   f"({prep_s:.1f}s, excluded)"),
        "seconds": dt, "host": cpu_info()}


def main():
    ap = argparse.ArgumentParser(description=__doc__,
                                 formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--replicas", type=int, default=4)
    ap.add_argument("--workload", default="mixtral_layer_decode_t1")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--cpu-tokens", type=int, default=16)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--glue", choices=("prenorm", "residual"), default="prenorm",
                    help="decode stacks: residual RMSNorm formed by each layer's router "
                         "(prenorm) or by a norm kernel after each layer (residual)")
    ap.add_argument("--graph", action="store_true",
                    help="stacks: replay one captured HIP graph per pass instead of launching each kernel")
    ap.add_argument("--pmc-pass", action="store_true",
                    help="warmup + timed decode steps only (for counter runs)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="plain 256 MiB device copy x5 (counter calibration)")
    ap.add_argument("--predictor", action="store_true",
                    help="time the Stacking Computer against sequential gates, p = 1..8")
    ap.add_argument("--loading", action="store_true",
                    help="expert loads host->HBM by precision, decode beside loads")
    ap.add_argument("--cache", action="store_true",
                    help="expert cache manager: policy miss penalties and replay rate (host only)")
    args = ap.parse_args()
    if args.cache:
        print(json.dumps(run_cache(args)), flush=True)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this library runs the layer on a "
              "single MI355X (no multi-GPU path); run with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    if args.copy_calibration:
        n = 256 << 20
        src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"mode": "copy-calibration", "bytes_read_per_launch": n,
                          "bytes_written_per_launch": n, "launches": 5}), flush=True)
        return
    import paper_2411_01433_amd as P
    P.lib()
    from synth import configs as C
    if args.predictor:
        print(json.dumps(run_predictor(args)), flush=True)
        return
    if args.loading:
        print(json.dumps(run_loading(args)), flush=True)
        return
    if C.BY_NAME[args.workload].n_layers > 1:
        out, state = run_stack(args)
        if not args.no_cpu_baseline and not args.pmc_pass:
            stack_cpu_baseline(args, state, out)
        print(json.dumps(out), flush=True)
        return
    out, state = run_decode_layer(args)
    if not args.no_cpu_baseline and not args.pmc_pass:
        parity_and_cpu(args, state, out)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
