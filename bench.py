#!/usr/bin/env python
"""Benchmark of the HSA operator on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input:
landmarks -> score + top-k -> forward -> backward (fwd+bwd workloads), or one decode step.
Inputs are resident in HBM before the timed region.  The main line is the 4K-context
fwd+bwd workload (B 8, L 4096, H 16 / G 2, d 128, S 64, k 8, bf16); under "also": the same
with the paper's main variant (stick-breaking weights, softmax off by one), the 64K-context
fwd+bwd, the wide-selection 16K workload (B 4, H 32 / G 4, S 128, k 16), the tiny fp32
workload (latency), the 1M-token decode step, and three layers sharing one selection over
inputs of its own (with, for comparison, a selection per layer).  Every fwd+bwd line
carries per-stage rates: landmarks and selection against HBM, forward and backward against
the bf16 matrix-core peak (fp32: the vector peak), from a pass with events between the four
calls; the decode line carries the scan against HBM and the attend stage.

Kernel durations come from HIP events recorded by the library around its launches on the
launch stream (hsa_attn_timing_enable / hsa_attn_timing_select).  The last warm-up step
brackets every kernel, which gives the per-kernel breakdown and the dominant kernel; the
timed steps bracket only that kernel (its roofline entry), so the other launches stay back
to back and the step time carries the cost of one event pair per step.  The decode step is
timed with no events; its per-kernel figures come from its warm-up.  The fp64 oracle is
timed on the host cores on a bounded sample (cpu_baseline).

Prints one JSON line.  `--gpus N` with N > 1 exits: this operator runs on one GPU.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "HSA fwd+bwd tokens/s at L=4K and 64K; decode µs/token at 1M-token ctx"

LABELS = {
    "L4K_bf16": "HSA fwd+bwd at 4K context: B8 L4096 H16/G2 d128 S64 k8, bf16",
    "L64K_bf16": "HSA fwd+bwd at 64K context: B1 L65536 H16/G2 d128 S64 k8, bf16",
    "wide_L16K_bf16": ("wide-selection HSA fwd+bwd: B4 L16384 H32/G4 d128 S128 k16, bf16; Q and "
                       "K of rank 16 plus N(0, 0.1) noise (many queries pick the same chunks)"),
    "tiny_f32": "tiny HSA fwd+bwd, fp32 (latency): B1 L1024 H4/G1 d64 S64 k4",
}

# MI355X published peaks
PEAK_HBM_GBS = 8000.0
PEAK_BF16_TFLOPS = 2500.0
PEAK_FP32_VALU_TFLOPS = 157.3

# per-kernel algorithmic work: ("flops" per valid (token, group, slot) pair in units of
# h*S*d, bound) or ("bytes", ...).  A valid pair is a selected chunk of a token.
# forward: Q K^T and P V (2 matmuls = 4 h S d flops); backward: 5 matmuls (recomputed
# Q K^T, dO V^T, (wP)^T dO, dz^T Q, dz K), all in the fused chunk pass, or split as
# Q K^T, dO V^T, dz K in the query pass and P^T dO, dz^T Q in the key pass.
MATMULS = {"forward_generic": 2, "forward_mfma": 2, "bwd_q_generic": 3, "bwd_q_mfma": 3,
           "bwd_kv_generic": 2, "bwd_kv_mfma": 2, "bwd_fused_mfma": 5, "fwd_chunk_mfma": 2}
MFMA_KERNELS = {"forward_mfma", "bwd_q_mfma", "bwd_kv_mfma", "bwd_fused_mfma", "fwd_chunk_mfma"}


def valid_pairs(B, L, G, S, k):
    """Number of (b, t, g, slot) with a selected chunk: sum_t min(k, floor(t/S))."""
    n = 0
    for c in range(-(-L // S)):
        rows = min(S, L - c * S)
        n += rows * min(k, c)
    return B * G * n


def kernel_work(name, sh, pairs):
    """(amount, unit, bound, peak) of the algorithmic work of one launch."""
    B, L, H, G, d, S, k = sh.B, sh.L, sh.H, sh.G, sh.d, sh.S, sh.k
    h = H // G
    es = 2 if sh.dtype == "bf16" else 4
    if name in MATMULS:
        fl = MATMULS[name] * 2.0 * h * S * d * pairs
        if name in MFMA_KERNELS:
            return fl, "TFLOP/s", "mfma", PEAK_BF16_TFLOPS
        return fl, "TFLOP/s", "alu", PEAK_FP32_VALU_TFLOPS
    C = L // S
    if name == "landmarks_kernel":
        return B * C * S * G * d * es + B * C * G * d * 4, "GB/s", "hbm", PEAK_HBM_GBS
    if name == "fwd_reduce":
        # reads each pair's partial output (h d bf16) and idx; writes O
        return (pairs * h * d * 2 + B * L * H * d * es + B * L * G * k * 4,
                "GB/s", "hbm", PEAK_HBM_GBS)
    if name == "bwd_dq_reduce":
        # reads each pair's partial dQ (h d bf16), Q, idx / w / dw; writes dQ, ds, q~
        return (pairs * h * d * 2 + 2 * B * L * H * d * es + B * L * G * k * 16 +
                B * L * G * d * 4, "GB/s", "hbm", PEAK_HBM_GBS)
    if name.startswith("select"):
        return (B * L * H * d * es + B * C * G * d * 4 + B * L * G * k * 8,
                "GB/s", "hbm", PEAK_HBM_GBS)
    return None


def make_training(name, torch):
    import hsa_synth
    wl = hsa_synth.WORKLOADS[name]
    sh = wl["shape"]
    t0 = time.time()
    inp = hsa_synth.make_training_inputs(name)
    dt = torch.bfloat16 if sh.dtype == "bf16" else torch.float32
    dev = {n: torch.from_numpy(v).to("cuda").to(dt) for n, v in inp.items()}
    return sh, inp, dev, time.time() - t0


def time_training(sh, dev, steps, warmup, torch, hsa, stick=False, off1=False):
    B, L, H, G, d, S, k = sh.B, sh.L, sh.H, sh.G, sh.d, sh.S, sh.k
    Q, K, V, dO = dev["Q"], dev["K"], dev["V"], dev["dO"]
    Kbar = torch.empty((B, L // S, G, d), dtype=torch.float32, device="cuda")
    idx = torch.empty((B, L, G, k), dtype=torch.int32, device="cuda")
    w = torch.empty((B, L, G, k), dtype=torch.float32, device="cuda")
    O = torch.empty_like(Q)
    grads = (torch.empty_like(Q), torch.empty_like(K), torch.empty_like(V))
    # the workspace depends on the variant (the off-by-one backward keeps more per pair)
    p = hsa.make_params(B, L, H, G, d, S, k, Q.dtype, stick_breaking=stick, off_by_one=off1)
    ws_f = torch.empty(max(1, hsa.workspace_size(p, hsa.HSA_OP_FORWARD)), dtype=torch.uint8,
                       device="cuda")
    ws_b = torch.empty(max(1, hsa.workspace_size(p, hsa.HSA_OP_BACKWARD)), dtype=torch.uint8,
                       device="cuda")

    stages = (
        ("landmarks", lambda: hsa.hsa_landmarks(K, S, out=Kbar)),
        ("select", lambda: hsa.hsa_select_topk(Q, Kbar, G, S, k, idx=idx, w=w,
                                               stick_breaking=stick)),
        ("forward", lambda: hsa.hsa_forward(Q, K, V, idx, w, S, out=O, workspace=ws_f,
                                            off_by_one=off1)),
        ("backward", lambda: hsa.hsa_backward(Q, K, V, Kbar, idx, w, dO, S, out=grads,
                                              workspace=ws_b, stick_breaking=stick,
                                              off_by_one=off1)))

    def step():
        for _, fn in stages:
            fn()

    ms, kern, brk = time_steps(step, steps, warmup, torch, hsa)
    return ms, kern, brk, stage_times(stages, max(2, min(steps, 5)), torch)


def gpu_backlog(torch, ms=2.0):
    """Queue about `ms` of device time ahead of the host (a spin kernel), so that launches
    enqueued next run back to back instead of waiting for the host; the spin is calibrated
    once per process."""
    global _SPIN_PER_MS
    if _SPIN_PER_MS is None:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(1000)                 # first launch of the spin kernel
        torch.cuda.synchronize()
        e0.record()
        torch.cuda._sleep(1000000)
        e1.record()
        torch.cuda.synchronize()
        _SPIN_PER_MS = 1000000 / max(e0.elapsed_time(e1), 1e-3)
    torch.cuda._sleep(int(ms * _SPIN_PER_MS))


_SPIN_PER_MS = None


def stage_times(stages, reps, torch):
    """Mean ms of each stage of a step, from events recorded between the stage calls on the
    current stream (a pass of its own, after the timed steps).  Each pass starts behind a
    queued spin kernel, so the events time the stages' kernels, not the host's calls."""
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(len(stages) + 1)]
    tot = [0.0] * len(stages)
    for _ in range(reps):
        gpu_backlog(torch)
        ev[0].record()
        for i, (_, fn) in enumerate(stages):
            fn()
            ev[i + 1].record()
        torch.cuda.synchronize()
        for i in range(len(stages)):
            tot[i] += ev[i].elapsed_time(ev[i + 1])
    return {name: tot[i] / reps for i, (name, _) in enumerate(stages)}


def candidate_scores(B, L, G, S):
    """Group scores a selection computes: sum over tokens of the candidate count."""
    n = 0
    for c in range(-(-L // S)):
        n += min(S, L - c * S) * c
    return B * G * n


def stage_fractions(sh, pairs, st):
    """Per stage: achieved rate of its algorithmic work and the fraction of the bound it
    meets (landmarks and selection against HBM, the attention stages against the matrix
    cores for bf16, the fp32 vector peak for fp32)."""
    B, L, H, G, d, S, k = sh.B, sh.L, sh.H, sh.G, sh.d, sh.S, sh.k
    h, C = H // G, L // S
    es = 2 if sh.dtype == "bf16" else 4
    mpeak, munit = ((PEAK_BF16_TFLOPS, "mfma") if sh.dtype == "bf16"
                    else (PEAK_FP32_VALU_TFLOPS, "alu"))
    work = {
        "landmarks": (B * C * S * G * d * es + B * C * G * d * 4, "hbm"),
        "select": (B * L * H * d * es + B * C * G * d * 4 + B * L * G * k * 8, "hbm"),
        "forward": (4.0 * h * S * d * pairs, munit),
        "backward": (10.0 * h * S * d * pairs, munit),
    }
    out = {}
    for name, ms in st.items():
        amount, bound = work[name]
        if bound == "hbm":
            rate = amount / (ms * 1e-3) / 1e9
            out[name] = {"ms": round(ms, 5), "bound": "hbm", "achieved": round(rate, 1),
                         "unit": "GB/s", "frac": round(rate / PEAK_HBM_GBS, 4),
                         "work": amount, "work_unit": "byte"}
        else:
            rate = amount / (ms * 1e-3) / 1e12
            peak = mpeak
            out[name] = {"ms": round(ms, 5), "bound": bound, "achieved": round(rate, 2),
                         "unit": "TFLOP/s", "frac": round(rate / peak, 4),
                         "work": amount, "work_unit": "flop"}
    out["select"]["score_flops"] = 2.0 * h * d * candidate_scores(B, L, G, S)
    return out


def bench_training(name, steps, warmup, torch, hsa, stick=False, off1=False, label=None):
    """One fwd+bwd workload: tokens/s, ms per step, per-kernel times, the roofline of the
    dominant kernel and the per-stage rates."""
    import hsa_synth
    sh, _, dev, _ = make_training(name, torch)
    ms, kern, brk, st = time_training(sh, dev, steps, warmup, torch, hsa, stick, off1)
    pairs = valid_pairs(sh.B, sh.L, sh.G, sh.S, sh.k)
    del dev
    torch.cuda.empty_cache()
    return {"workload": label or hsa_synth.WORKLOADS[name].get("label", name),
            "tokens_per_s": round(sh.B * sh.L / (ms * 1e-3), 1), "ms_per_step": round(ms, 4),
            "roofline": roofline_of(kern, sh, pairs, name),
            "stages": stage_fractions(sh, pairs, st),
            "kernels_avg_ms": {n: round(t / c, 5) for n, (c, t) in brk.items()}}


def time_steps(step, steps, warmup, torch, hsa):
    """(ms per step, roofline-kernel timings of the timed steps, per-kernel breakdown)."""
    # Untimed warm-up; its last step brackets every kernel (the per-kernel breakdown and
    # the dominant kernel).  The timed steps bracket only the dominant kernel: an event pair
    # costs queue time between launches, which would otherwise count in the step time.
    hsa.timing_enable(False)
    hsa.timing_select(None)
    for i in range(warmup):
        if i == warmup - 1:
            torch.cuda.synchronize()
            hsa.timing_collect()               # drop anything recorded before
            gpu_backlog(torch)                 # the step's launches then run back to back
            hsa.timing_enable(True)
        step()
    torch.cuda.synchronize()
    hsa.timing_enable(False)
    breakdown = hsa.timing_collect() if warmup else {}
    dominant = max(breakdown.items(), key=lambda kv: kv[1][1])[0] if breakdown else None
    hsa.timing_select(dominant)                # None: every kernel
    hsa.timing_enable(True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    hsa.timing_enable(False)
    hsa.timing_select(None)
    kern = hsa.timing_collect()
    ms = e0.elapsed_time(e1) / steps
    return ms, kern, breakdown or kern


def source_digest():
    """sha256 over the HIP sources and headers of the library (traffic figures measured on
    other sources are stale)."""
    import glob
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2504_16795_amd", "csrc")
    for f in sorted(glob.glob(os.path.join(csrc, "*.hip")) + glob.glob(os.path.join(csrc, "*.h"))):
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def traffic_of(name, workload):
    """HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, calibrated) of `name` on `workload`
    from profiles/traffic_<workload>.json, or None if absent or taken on other sources."""
    path = os.path.join(ROOT, "profiles", "traffic_%s.json" % workload)
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh)
    if rec.get("source_sha256") != source_digest():
        return None
    k = rec.get("kernels", {}).get(name)
    return None if k is None else k["hbm_bytes_per_launch"]


def roofline_of(kern, sh, pairs, workload):
    """Roofline entry of the kernel with the largest total time in the timed region."""
    name, (cnt, tot) = max(kern.items(), key=lambda kv: kv[1][1])
    work = kernel_work(name, sh, pairs)
    avg_ms = tot / cnt
    if work is None:
        return {"kernel": name, "avg_ms": avg_ms, "bound": None}
    amount, unit, bound, peak = work
    if unit == "TFLOP/s":
        achieved = amount / (avg_ms * 1e-3) / 1e12
    else:
        achieved = amount / (avg_ms * 1e-3) / 1e9
    return {"kernel": name, "bound": bound, "achieved": round(achieved, 3), "peak": peak,
            "unit": unit, "frac": round(achieved / peak, 5),
            "traffic": traffic_of(name, workload),
            "avg_ms": round(avg_ms, 5), "launches": cnt,
            "work_per_launch": amount,
            "work_unit": "flop" if unit == "TFLOP/s" else "byte"}


def bench_decode(steps, warmup, torch, hsa):
    import hsa_synth
    wl = hsa_synth.WORKLOADS["decode_1M_bf16"]
    sh = wl["shape"]
    inp = hsa_synth.make_decode_inputs(sh, wl["seed"], device="cuda")
    q, Kc, Vc = inp["q"], inp["Kc"], inp["Vc"]
    kbar = hsa.hsa_landmarks(Kc, sh.S, kbar_dtype=torch.bfloat16)
    p = hsa.make_params(sh.B, sh.L, sh.H, sh.G, sh.d, sh.S, sh.k, q.dtype)
    ws = torch.empty(hsa.workspace_size(p, hsa.HSA_OP_DECODE), dtype=torch.uint8, device="cuda")
    o = torch.empty_like(q)
    idx = torch.empty((sh.B, sh.G, sh.k), dtype=torch.int32, device="cuda")
    w = torch.empty((sh.B, sh.G, sh.k), dtype=torch.float32, device="cuda")
    # warm-up (its second half with every kernel bracketed: the per-kernel figures), then
    # timed steps with no events between the launches
    hsa.timing_select(None)
    for i in range(warmup):
        if i == warmup // 2:
            torch.cuda.synchronize()
            hsa.timing_collect()
            gpu_backlog(torch, 0.1 * warmup + 1.0)
            hsa.timing_enable(True)
        hsa.hsa_decode(q, Kc, Vc, kbar, sh.S, sh.k, out=(o, idx, w), workspace=ws)
    torch.cuda.synchronize()
    hsa.timing_enable(False)
    kern = hsa.timing_collect()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(backlog):
        # backlog: the steps queued behind a spin kernel, so that the events time the
        # device's work alone (back to back, as a captured graph would run it); without it,
        # the host's calls pace the steps
        torch.cuda.synchronize()
        if backlog:
            gpu_backlog(torch, 0.1 * steps + 1.0)
        e0.record()
        for _ in range(steps):
            hsa.hsa_decode(q, Kc, Vc, kbar, sh.S, sh.k, out=(o, idx, w), workspace=ws)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps * 1e3

    us = timed(True)
    us_host = timed(False)
    planted_ok = all(int(inp["planted"][b, g]) in idx[b, g].tolist()
                     for b in range(sh.B) for g in range(sh.G))
    C = sh.L // sh.S
    stream_bytes = sh.B * C * sh.G * sh.d * 2                     # bf16 landmark cache
    gather_bytes = sh.B * sh.G * sh.k * sh.S * sh.d * 2 * 2       # selected K and V chunks
    scan = kern.get("decode_scan")
    out = {"workload": "decode 1M ctx: B8, 1 token/seq, cache 2^20 tokens (16384 chunks of 64),"
                       " H16/G2 d128 k8, bf16 landmark cache",
           "us_per_step": round(us, 3), "us_per_sequence_token": round(us / sh.B, 3),
           "us_per_step_host_paced": round(us_host, 3),
           "timing": ("us_per_step: the steps' device time, queued back to back behind a spin "
                      "kernel; us_per_step_host_paced: the same steps launched as the host "
                      "makes the calls"),
           "tokens_per_s": round(sh.B / (us * 1e-6), 1), "planted_chunk_selected": planted_ok,
           "kernels_avg_us": {n: round(t / c * 1e3, 3) for n, (c, t) in kern.items()},
           "kernels_timed_in": "second half of the warm-up (event pairs around each launch)"}
    if scan:
        avg = scan[1] / scan[0]
        gbs = stream_bytes / (avg * 1e-3) / 1e9
        out["scan_roofline"] = {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS,
                                "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
                                "bytes_per_launch": stream_bytes,
                                "traffic": traffic_of("decode_scan", "decode_1M_bf16")}
    out["algorithmic_bytes_per_step"] = stream_bytes + gather_bytes
    # per stage: the scan streams the landmark cache (HBM-bound); the attend stage (merge,
    # attention, combine) reads the selected chunks' keys and values
    att = [kern[n] for n in ("decode_attend_mfma", "decode_combine", "decode_finish") if n in kern]
    stages = {}
    if scan:
        stages["scan"] = dict(out["scan_roofline"], us=round(scan[1] / scan[0] * 1e3, 3))
    if att:
        us_att = sum(t / c for c, t in att) * 1e3
        gbs = gather_bytes / (us_att * 1e-6) / 1e9
        stages["attend"] = {"us": round(us_att, 3), "bound": "hbm", "achieved": round(gbs, 1),
                            "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
                            "bytes_per_step": gather_bytes}
    out["stages"] = stages
    # the same step with the key / value cache in pinned host memory: only the landmark
    # cache stays on the GPU, and the selected chunks cross the host link each step
    Kh = torch.empty(Kc.shape, dtype=Kc.dtype, pin_memory=True)
    Vh = torch.empty(Vc.shape, dtype=Vc.dtype, pin_memory=True)
    Kh.copy_(Kc)
    Vh.copy_(Vc)
    wsh = torch.empty(hsa.workspace_size(p, hsa.HSA_OP_DECODE_HOST), dtype=torch.uint8,
                      device="cuda")
    oh, idxh, wh = torch.empty_like(o), torch.empty_like(idx), torch.empty_like(w)
    for i in range(warmup):
        if i == warmup // 2:
            torch.cuda.synchronize()
            hsa.timing_collect()
            gpu_backlog(torch, 0.1 * warmup + 1.0)
            hsa.timing_enable(True)
        hsa.hsa_decode_host(q, Kh, Vh, kbar, sh.S, sh.k, out=(oh, idxh, wh), workspace=wsh)
    torch.cuda.synchronize()
    hsa.timing_enable(False)
    kern_h = hsa.timing_collect()
    e0.record()
    for _ in range(steps):
        hsa.hsa_decode_host(q, Kh, Vh, kbar, sh.S, sh.k, out=(oh, idxh, wh), workspace=wsh)
    e1.record()
    torch.cuda.synchronize()
    us_h = e0.elapsed_time(e1) / steps * 1e3
    host = {"us_per_step": round(us_h, 3), "us_per_sequence_token": round(us_h / sh.B, 3),
            "same_outputs_as_device_cache": bool(torch.equal(oh, o) and torch.equal(idxh, idx)
                                                 and torch.equal(wh, w)),
            "kernels_avg_us": {n: round(t / c * 1e3, 3) for n, (c, t) in kern_h.items()},
            "host_bytes_per_step": gather_bytes,
            "gpu_resident_bytes": stream_bytes}
    ga = kern_h.get("decode_gather")
    if ga:
        host["gather_GBps"] = round(gather_bytes / (ga[1] / ga[0] * 1e-3) / 1e9, 1)
    out["host_kv_cache"] = host
    del Kh, Vh
    return out


def bench_shared(steps, warmup, torch, hsa):
    """Sec. 4.4's setting: three attention layers sharing one selection over inputs of their
    own (d_sel = h d_h = 1024), forward and backward of all three plus the selection and its
    backward per step; and the same with a selection (and its backward) per layer."""
    import hsa_synth
    sh = hsa_synth.WORKLOADS["shared_x3_L4K_bf16"]["shape"]
    B, L, H, G, d, S, k = sh.B, sh.L, sh.H, sh.G, sh.d, sh.S, sh.k
    dsel = (H // G) * d
    layers, Qs, Ks = hsa_synth.make_shared_selection_inputs("shared_x3_L4K_bf16")
    idx = torch.empty((B, L, G, k), dtype=torch.int32, device="cuda")
    w = torch.empty((B, L, G, k), dtype=torch.float32, device="cuda")
    dw = torch.empty_like(w)
    O = torch.empty_like(layers[0]["Q"])
    grads = (torch.empty_like(layers[0]["Q"]), torch.empty_like(layers[0]["K"]),
             torch.empty_like(layers[0]["V"]))
    sel_grads = (torch.empty_like(Qs), torch.empty_like(Ks))
    p = hsa.make_params(B, L, H, G, d, S, k, torch.bfloat16)
    ps = hsa.make_params(B, L, G, G, dsel, S, k, torch.bfloat16)
    ws_f = torch.empty(max(1, hsa.workspace_size(p, hsa.HSA_OP_FORWARD)), dtype=torch.uint8,
                       device="cuda")
    ws_b = torch.empty(max(1, hsa.workspace_size(p, hsa.HSA_OP_BACKWARD)), dtype=torch.uint8,
                       device="cuda")
    ws_s = torch.empty(max(1, hsa.workspace_size(ps, hsa.HSA_OP_SELECT_BACKWARD)),
                       dtype=torch.uint8, device="cuda")

    def shared():
        hsa.hsa_select_topk(Qs, Ks, G, S, k, idx=idx, w=w)
        for lay in layers:
            hsa.hsa_forward(lay["Q"], lay["K"], lay["V"], idx, w, S, out=O, workspace=ws_f)
        for i, lay in enumerate(layers):
            hsa.hsa_backward_attn(lay["Q"], lay["K"], lay["V"], idx, w, lay["dO"], S, out=grads,
                                  dw=dw, accumulate_dw=i > 0, workspace=ws_b)
        hsa.hsa_select_backward(Qs, Ks, idx, w, dw, G, S, out=sel_grads, workspace=ws_s)

    def per_layer():
        for lay in layers:
            hsa.hsa_select_topk(Qs, Ks, G, S, k, idx=idx, w=w)
            hsa.hsa_forward(lay["Q"], lay["K"], lay["V"], idx, w, S, out=O, workspace=ws_f)
        for lay in layers:
            hsa.hsa_backward_attn(lay["Q"], lay["K"], lay["V"], idx, w, lay["dO"], S, out=grads,
                                  dw=dw, workspace=ws_b)
            hsa.hsa_select_backward(Qs, Ks, idx, w, dw, G, S, out=sel_grads, workspace=ws_s)

    ms, _, brk = time_steps(shared, steps, warmup, torch, hsa)
    ms_pl, _, _ = time_steps(per_layer, steps, warmup, torch, hsa)
    return {"workload": ("3 HSA layers sharing one selection at 4K context: B8 L4096 H16/G2 "
                         "d128 S64 k8, selection inputs d_sel 1024, bf16; fwd+bwd of the "
                         "3 layers, the selection and its backward"),
            "tokens_per_s": round(B * L / (ms * 1e-3), 1), "ms_per_step": round(ms, 4),
            "ms_per_step_selection_per_layer": round(ms_pl, 4),
            "kernels_avg_ms": {n: round(t / c, 5) for n, (c, t) in brk.items()}}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(name, inp, budget_s=12.0, max_slices=16):
    """Oracle fwd+bwd on whole (b, g) slices of the workload until the budget is used, each
    stage timed on its own."""
    import numpy as np
    import hsa_synth
    import oracle
    sh = hsa_synth.WORKLOADS[name]["shape"]
    L, G, h, d, S, k = sh.L, sh.G, sh.H // sh.G, sh.d, sh.S, sh.k
    oracle.build(force=False)
    done, t0 = 0, time.time()
    st = {"landmarks": 0.0, "select": 0.0, "forward": 0.0, "backward": 0.0}

    def timed(stage, fn, *a):
        t = time.time()
        r = fn(*a)
        st[stage] += time.time() - t
        return r

    for b in range(sh.B):
        for g in range(G):
            dm = oracle.dims(L, h, d, S, k)
            Qs = np.ascontiguousarray(inp["Q"][b, :, g * h:(g + 1) * h], dtype=np.float64)
            dOs = np.ascontiguousarray(inp["dO"][b, :, g * h:(g + 1) * h], dtype=np.float64)
            Ks = np.ascontiguousarray(inp["K"][b, :, g], dtype=np.float64)
            Vs = np.ascontiguousarray(inp["V"][b, :, g], dtype=np.float64)
            Kb = timed("landmarks", oracle.landmarks_slice, dm, Ks)
            idx, w, _, _ = timed("select", oracle.select_slice, dm, Qs, Kb)
            timed("forward", oracle.forward_slice, dm, Qs, Ks, Vs, idx, w)
            _, ds = timed("backward", oracle.backward_q_slice, dm, Qs, Ks, Vs, Kb, idx, w, dOs)
            timed("backward", oracle.backward_kv_slice, dm, Qs, Ks, Vs, idx, w, dOs, ds)
            done += 1
            if time.time() - t0 >= budget_s or done >= max_slices:
                break
        if time.time() - t0 >= budget_s or done >= max_slices:
            break
    el = time.time() - t0
    tokens = done * L / G            # each (b, g) slice is 1/G of a sequence's work
    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or os.cpu_count()
    return {"value": round(tokens / el, 2), "unit": "tokens/s", "cores": threads,
            "kind": "oracle", "cpu_model": cpu_model(),
            "stage_seconds": {n: round(v, 3) for n, v in st.items()},
            "stage_tokens_per_s": {n: round(tokens / v, 1) for n, v in st.items() if v > 0},
            "sample": "%d of %d (batch, group) slices of the %s workload, fwd+bwd "
                      "(landmarks, select, forward, backward), fp64 on %d OpenMP threads, "
                      "%.1f s" % (done, sh.B * G, name, threads, el)}


CALIB_BYTES = 256 << 20


def pmc_run(workload, steps, torch, hsa):
    """Workload for counter collection under rocprofv3 --pmc: a device copy of CALIB_BYTES
    (the calibration of FETCH_SIZE / WRITE_SIZE) three times, then `steps` steps."""
    x = torch.empty(CALIB_BYTES // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    y = torch.empty_like(x)
    for _ in range(3):
        y.copy_(x)
    torch.cuda.synchronize()
    if workload == "decode_1M_bf16":
        # the cache set-up (one landmark launch over the whole cache), then `steps` decode
        # steps with the cache in HBM and `steps` with it in host memory
        bench_decode(steps, 0, torch, hsa)
    else:
        sh, _, dev, _ = make_training(workload, torch)
        time_training(sh, dev, steps, 1, torch, hsa)
    torch.cuda.synchronize()


def pmc_summarize(workload, fetch_csv, write_csv, out_path):
    """Per-kernel HBM traffic from the two counter passes, calibrated on the copy kernel:
    factor = bytes the copy moves / bytes the counter reports for it."""
    import csv
    from collections import defaultdict

    def read(path, counter):
        per = defaultdict(list)
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"].startswith(counter):
                per[r["Kernel_Name"]].append((int(r["Dispatch_Id"]),
                                              float(r["Counter_Value"]) * 1024.0))   # KiB
        return {n: [v for _, v in sorted(x)] for n, x in per.items()}

    fetch, write = read(fetch_csv, "FETCH_SIZE"), read(write_csv, "WRITE_SIZE")
    # the runtime's device-to-device copy kernel (torch's same-dtype copy_ goes through it)
    copy = [n for n in fetch if "copybuffer" in n.lower()]
    if not copy:
        raise SystemExit("no copy kernel in %s" % fetch_csv)
    # the calibration copies are the first three dispatches of that kernel (a workload may
    # copy more later, e.g. the decode workload's device-to-host copy of its cache)
    cname = max(copy, key=lambda n: max(fetch[n][:3]))
    f_fac = CALIB_BYTES / sorted(fetch[cname][:3])[1]
    w_fac = CALIB_BYTES / sorted(write[cname][:3])[1]
    # function-name fragment -> the name the library's timing reports
    names = {"landmarks_kernel": "landmarks_kernel", "select_tiles_kernel": "select_kernel",
             "select_split_kernel": "select_kernel", "select_kernel": "select_kernel",
             "select_mfma": "select_kernel",
             "forward_mfma": "forward_mfma", "bwd_q_mfma": "bwd_q_mfma",
             "bwd_kv_mfma": "bwd_kv_mfma", "bitmap_build": "bitmap_build",
             "bwd_fused_mfma": "bwd_fused_mfma", "bwd_dq_reduce": "bwd_dq_reduce",
             "bwd_lmk_stream": "bwd_lmk_stream", "bwd_finish": "bwd_finish",
             "bwd_rowcount": "bwd_plan", "bwd_plan": "bwd_plan",
             "fwd_chunk_mfma": "fwd_chunk_mfma", "fwd_reduce": "fwd_reduce",
             "stream_rowcount": "plan", "stream_plan": "plan",
             "forward_generic": "forward_generic",
             "bwd_q_generic": "bwd_q_generic", "bwd_kv_generic": "bwd_kv_generic",
             "decode_scan": "decode_scan", "decode_attend_mfma": "decode_attend_mfma",
             "decode_gather": "decode_gather", "decode_finish": "decode_finish",
             "decode_combine": "decode_combine", "decode_attend_slot": "decode_attend_mfma",
             "bwd_kv_finish": "bwd_kv_finish", "kv_generic_finish": "bwd_kv_finish"}
    # per timing name: the bytes of every kernel that maps to it (the two plan kernels, say,
    # each launched once per step) summed, per launch of the stage (the largest dispatch
    # count among them); per full kernel name as well
    totals, by_kernel = {}, {}
    for full in fetch:
        short = next((v for n, v in names.items() if n in full), None)
        if short is None or full not in write:
            continue
        ft, wt, nd = sum(fetch[full]) * f_fac, sum(write[full]) * w_fac, len(fetch[full])
        by_kernel[full] = {"short": short, "fetch_bytes_per_launch": round(ft / nd),
                           "write_bytes_per_launch": round(wt / nd), "dispatches": nd}
        t = totals.setdefault(short, [0.0, 0.0, 0])
        t[0] += ft
        t[1] += wt
        t[2] = max(t[2], nd)
    kernels = {}
    for short, (ft, wt, nd) in totals.items():
        fb, wb = ft / nd, wt / nd
        kernels[short] = {"fetch_bytes_per_launch": round(fb), "write_bytes_per_launch": round(wb),
                          "hbm_bytes_per_launch": round(fb + wb), "dispatches": nd}
    rec = {"workload": workload, "source_sha256": source_digest(),
           "calibration": {"kernel": cname, "bytes": CALIB_BYTES,
                           "fetch_factor": round(f_fac, 4), "write_factor": round(w_fac, 4)},
           "kernels": kernels, "by_kernel": by_kernel}
    with open(out_path, "w") as fh:
        json.dump(rec, fh, indent=1)
    print(json.dumps(rec))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the 64K fwd+bwd and 1M decode lines")
    ap.add_argument("--pmc-run", metavar="WORKLOAD",
                    help="calibration copy + a few steps of WORKLOAD, for rocprofv3 --pmc")
    ap.add_argument("--pmc-summarize", nargs=4,
                    metavar=("WORKLOAD", "FETCH_CSV", "WRITE_CSV", "OUT_JSON"),
                    help="turn the two counter passes into profiles/traffic_<workload>.json")
    args = ap.parse_args()
    if args.pmc_summarize:
        pmc_summarize(*args.pmc_summarize)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py: the HSA operator here is a single-GPU build; run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2504_16795_amd as hsa
    hsa.load()
    torch.cuda.init()
    if args.pmc_run:
        pmc_run(args.pmc_run, 3, torch, hsa)
        return

    name = "L4K_bf16"
    sh, inp, dev, gen_s = make_training(name, torch)
    print("[bench] %s inputs ready (%.1f s)" % (name, gen_s), file=sys.stderr, flush=True)
    ms, kern, brk, st = time_training(sh, dev, args.steps, args.warmup, torch, hsa)
    pairs = valid_pairs(sh.B, sh.L, sh.G, sh.S, sh.k)
    tokens = sh.B * sh.L
    res = {
        "metric": METRIC, "value": round(tokens / (ms * 1e-3), 1), "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": LABELS[name],
                   "batch": sh.B, "seq_len": sh.L, "q_heads": sh.H, "kv_heads": sh.G,
                   "head_dim": sh.d, "chunk": sh.S, "topk": sh.k},
        "roofline": roofline_of(kern, sh, pairs, name),
        "stages": stage_fractions(sh, pairs, st),
        "kernels_avg_ms": {n: round(t / c, 5) for n, (c, t) in brk.items()},
        "kernels_timed_in": ("last warm-up step (event pairs around each launch); the timed "
                             "steps bracket only the roofline kernel; stages from a pass of "
                             "their own with events between the four calls"),
    }
    print("[bench] %s: %.3f ms/step" % (name, ms), file=sys.stderr, flush=True)
    del dev
    torch.cuda.empty_cache()
    if not args.no_extra:
        also = res["also"] = {}
        # the paper's main variant on the same workload: stick-breaking chunk weights and
        # the softmax off by one inside a chunk
        also["L4K_bf16_main_variant"] = bench_training(
            name, max(2, args.steps // 2), 2, torch, hsa, stick=True, off1=True,
            label=LABELS[name] + "; stick-breaking weights and softmax off by one")
        print("[bench] %s main variant: %.3f ms/step"
              % (name, also["L4K_bf16_main_variant"]["ms_per_step"]), file=sys.stderr, flush=True)
        for extra in ("L64K_bf16", "wide_L16K_bf16", "tiny_f32"):
            also[extra] = bench_training(extra, max(2, args.steps // 2), 2, torch, hsa,
                                         label=LABELS[extra])
            print("[bench] %s: %.3f ms/step" % (extra, also[extra]["ms_per_step"]),
                  file=sys.stderr, flush=True)
        also["decode_1M_bf16"] = bench_decode(max(20, args.steps * 5), 10, torch, hsa)
        print("[bench] decode: %.2f us/step" % also["decode_1M_bf16"]["us_per_step"],
              file=sys.stderr, flush=True)
        torch.cuda.empty_cache()
        also["shared_x3_L4K_bf16"] = bench_shared(max(2, args.steps // 2), 2, torch, hsa)
        print("[bench] shared selection x3: %.3f ms/step"
              % also["shared_x3_L4K_bf16"]["ms_per_step"], file=sys.stderr, flush=True)
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(name, inp)
        print("[bench] cpu baseline done", file=sys.stderr, flush=True)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
