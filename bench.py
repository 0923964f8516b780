#!/usr/bin/env python3
"""Throughput of the fused attention-distillation KL on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input:
the forward (streamkl_fwd: KL, LSE1, LSE2 for every row) followed by the
standard-distillation backward (streamkl_bwd: dQ2 via the query-owned kernel,
then dK2 via the key-owned kernel) with the paper's mean objective
(dkl = 1 / (B H N_Q)). Inputs are resident in HBM before timing starts.

Workload (the one the 16K figure is quoted on): B=1, H=32, N_Q=N_K=16384,
d1=d2=128, s=1/sqrt(128), non-causal, student Q2 = bf16(Q1 + 0.3 eps), K2 = K1.
Prints ONE JSON line.

Timing (the method of the measurement plan):
  * `value` / `ms_per_step`: wall clock over K back-to-back steps, bracketed
    by device synchronisation, after W warm-up steps.
  * per-kernel figures: HIP events on the launch stream around each kernel,
    over `--reps` further steps (at least 10 at 64K); before every one of
    them a 512 MiB buffer is written, which evicts the 256 MB last-level
    cache (MALL), so no step finds the previous one's tiles there. Median and
    minimum are reported.
  * algorithmic work: 2 (d1 + d2) flop per unmasked pair forward and
    (2 d1 + 6 d2) flop per pair for the student backward, the recompute of
    S1 and S2 counted once (the fused ideal). Of it, each of the two separate
    backward kernels is credited its own gradient contraction (2 d2) and half
    the recompute (d1 + d2). The work each kernel actually executes (the
    recompute in both) is reported beside it as "own work".
  * `roofline`: the dominant kernel (largest median) under that accounting;
    `roofline_target` is the forward (the 50%-of-peak target row),
    `roofline_bwd_pass` the two backward kernels together.
  * `mfma_peak`: back-to-back bf16 MFMA throughput of this chip on N(0,1)
    and on constant operands (libstreamkl_bench.so), so that every fraction of
    the published 2500 TFLOP/s also appears as a fraction of what the MFMA
    units sustain on random data at the clock the box runs.
  * `cpu_baseline`: the fp64 oracle (not the target) on a bounded sample of
    the same workload, in a process pool on the host's cores, run before the
    GPU is touched.

Side sections (each can be switched off): the 64K causal long-context
workload ("long_context"), the other causal workloads ("workloads"), the
split-K forward and the backward strategies on decode-like shapes
("split_k", "fused_bwd"), the sigmoid-score path ("sigmoid") and the clock
probe ("clock_probe").

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--reps R] [--no-64k] [--no-cpu-baseline]
                    [--no-split] [--no-fused] [--no-workloads] [--no-clock-probe] [--no-mfma-peak] [--no-sigmoid]
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBPS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.json")
EVICT_BYTES = 512 << 20        # twice the 256 MB MALL
KERNEL_NAMES = {"fwd": "kl_fwd_kernel<128,128>", "dq": "kl_bwd_dq_kernel<128,128,mode1>",
                "dk": "kl_bwd_dk_kernel<128,128,mode1>"}


def kernel_source_hash():
    """SHA-256 over the code of the HIP sources and the C header: counters are only valid for the code they
    measured. Comments and layout are left out, so editing a comment keeps the measurement."""
    import glob
    import hashlib
    import re
    h = hashlib.sha256()
    files = sorted(glob.glob(os.path.join(ROOT, "paper_2606_20005_amd", "csrc", "*.h*"))) + \
        [os.path.join(ROOT, "include", "streamkl.h")]
    for f in files:
        with open(f, "rb") as fh:
            text = fh.read()
        text = re.sub(rb"/\*.*?\*/", b" ", text, flags=re.S)
        text = re.sub(rb"//[^\n]*", b"", text)
        h.update(os.path.basename(f).encode() + b"\0" + b" ".join(text.split()))
    return h.hexdigest()


def measured_traffic(kernel):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 FETCH_SIZE / WRITE_SIZE passes,
    scaled by the copy-kernel calibration; None if absent or taken on different kernel sources."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("csrc_sha256") != kernel_source_hash():
        return None
    k = t.get("kernels", {}).get(kernel)
    return None if k is None else int(k["hbm_bytes"])


def pairs(w, causal):
    """Unmasked (query, key) pairs: the unit every per-pair figure is multiplied by."""
    if not causal:
        return w.B * w.H * w.n_q * w.n_k
    nq, nk = w.n_q, w.n_k
    full = max(0, nk - nq)          # bottom-right alignment (n_q <= n_k here)
    return w.B * w.H * (nq * full + nq * (nq + 1) // 2)


def flops_per_pair(d1, d2):
    """Algorithmic flop per unmasked pair: the recompute counted once over the backward, half credited to
    each separate backward kernel; "own" is what each kernel executes."""
    return {
        "fwd": 2 * (d1 + d2),
        "dq": (d1 + d2) + 2 * d2,
        "dk": (d1 + d2) + 2 * d2,
        "bwd": 2 * (d1 + d2) + 4 * d2,
        "own": {"fwd": 2 * (d1 + d2), "dq": 2 * (d1 + d2) + 2 * d2, "dk": 2 * (d1 + d2) + 2 * d2},
    }


def upload(d):
    import numpy as np
    import torch
    from paper_2606_20005_amd import inputs
    out = []
    for k in ("Q1", "K1", "Q2", "K2"):
        out.append(torch.from_numpy(inputs.bf16_bits(d[k]).view(np.int16)).view(torch.bfloat16).cuda())
        del d[k]
    return out


class Evictor:
    """Before a timed rep: writes EVICT_BYTES of device memory, then reads another EVICT_BYTES buffer. The write
    displaces the workload's data from the MALL; the read displaces the write's dirty lines, so that their write-back
    to HBM happens here and not inside the timed kernel (a write alone cost the HBM-bound decode kernels a third of
    their bandwidth). Afterwards the MALL holds none of the workload's data and no dirty lines."""

    def __init__(self):
        import torch
        self.buf = torch.empty(EVICT_BYTES // 4, dtype=torch.float32, device="cuda")
        self.clean = torch.ones(EVICT_BYTES // 4, dtype=torch.float32, device="cuda")
        self.k = 0

    def __call__(self):
        self.k += 1
        self.buf.fill_(float(self.k))
        self.clean.sum()


def run_workload(sk, w, causal, steps, warmup, reps, evict):
    """Wall ms per step over `steps` back-to-back steps, then per-kernel event times (ms) over `reps` steps,
    each after a cache eviction (Evictor). Returns (wall_ms, {kernel: [ms, ...]}, extra, kl_mean)."""
    import torch
    from paper_2606_20005_amd import inputs
    d = inputs.make(w)
    q1, k1, q2, k2 = upload(d)
    B, H, NQ, NK = w.B, w.H, w.n_q, w.n_k
    dev = q1.device
    kl, l1, l2 = (torch.empty((B, H, NQ), dtype=torch.float32, device=dev) for _ in range(3))
    g = torch.full((B, H, NQ), 1.0 / (B * H * NQ), dtype=torch.float32, device=dev)
    dq2 = torch.empty((B, H, NQ, w.d2), dtype=torch.float32, device=dev)
    dk2 = torch.empty((B, H, NK, w.d2), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        sk.fwd(q1, k1, q2, k2, w.s1, w.s2, causal, 0, out=(kl, l1, l2))
        if ev is not None:
            ev[1].record(stream)
        sk.bwd(q1, k1, q2, k2, kl, l1, l2, g, w.s1, w.s2, causal, 0, want=("dq2", "dk2"),
               out={"dq2": dq2, "dk2": dk2})
        if ev is not None:
            ev[2].record(stream)

    def dq_alone(ev):
        ev[3].record(stream)
        sk.bwd(q1, k1, q2, k2, kl, l1, l2, g, w.s1, w.s2, causal, 0, want=("dq2",), out={"dq2": dq2})
        ev[4].record(stream)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    free0, _ = torch.cuda.mem_get_info()
    alloc0 = torch.cuda.max_memory_allocated()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3 / steps
    free1, _ = torch.cuda.mem_get_info()
    # One step: the forward, then one backward call for dQ2 and dK2 (the dK
    # kernel first, streaming row statistics prepared into the dQ2 output,
    # then the dQ kernel). The dQ kernel is timed alone by a dQ2-only call
    # after another eviction; the dK kernel (with its statistics prep) is the
    # two-gradient call less that, rep by rep.
    times = {"fwd": [], "dq": [], "dk": [], "bwd": []}
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(reps)]
    for r in range(reps):
        evict()
        step(events[r])
        evict()
        dq_alone(events[r])
    torch.cuda.synchronize()
    for ev in events:
        bwd = ev[1].elapsed_time(ev[2])
        dq = ev[3].elapsed_time(ev[4])
        times["fwd"].append(ev[0].elapsed_time(ev[1]))
        times["bwd"].append(bwd)
        times["dq"].append(dq)
        times["dk"].append(bwd - dq)
    extra = {
        "workspace_bytes": 0,
        "stats_bytes": 12 * B * H * NQ,
        "grad_output_bytes": int(dq2.numel() + dk2.numel()) * 4,
        "device_free_delta_bytes": int(free0 - free1),
        "torch_peak_alloc_delta_bytes": int(torch.cuda.max_memory_allocated() - alloc0),
    }
    kl_mean = float(kl.mean())
    del q1, k1, q2, k2, kl, l1, l2, g, dq2, dk2
    torch.cuda.empty_cache()
    return wall_ms, times, extra, kl_mean


def summarize(w, causal, times, peak_measured=None):
    """Per-kernel median/min ms, algorithmic and own-work TFLOP/s, fractions of the bf16 peak."""
    P = pairs(w, causal)
    f = flops_per_pair(w.d1, w.d2)
    out = {}
    for k in ("fwd", "dq", "dk"):
        med, mn = statistics.median(times[k]), min(times[k])
        tf = f[k] * P / (med * 1e-3) / 1e12
        out[k] = {"ms_median": round(med, 4), "ms_min": round(mn, 4), "reps": len(times[k]),
                  "flop_per_launch": f[k] * P, "tflops": round(tf, 2),
                  "frac_bf16_peak": round(tf / PEAK_BF16_TFLOPS, 4),
                  "own_work_flop_per_launch": f["own"][k] * P,
                  "own_work_tflops": round(f["own"][k] * P / (med * 1e-3) / 1e12, 2)}
        if peak_measured:
            out[k]["frac_measured_peak"] = round(tf / peak_measured, 4)
    bwd_med = statistics.median(times["bwd"])
    tf = f["bwd"] * P / (bwd_med * 1e-3) / 1e12
    out["bwd"] = {"ms_median": round(bwd_med, 4), "flop": f["bwd"] * P, "tflops": round(tf, 2),
                  "frac_bf16_peak": round(tf / PEAK_BF16_TFLOPS, 4)}
    if peak_measured:
        out["bwd"]["frac_measured_peak"] = round(tf / peak_measured, 4)
    return out, P, f


def mfma_peak_figures(reps=5, iters=20000):
    """Back-to-back bf16 MFMA throughput on N(0,1) and on all-ones operands (libstreamkl_bench.so)."""
    import ctypes
    import torch
    path = os.path.join(ROOT, "paper_2606_20005_amd", "libstreamkl_bench.so")
    lib = ctypes.CDLL(path)
    lib.streamkl_bench_mfma_peak.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                             ctypes.c_void_p]
    lib.streamkl_bench_mfma_peak.restype = ctypes.c_int
    waves = 256 * 4                # one wave per SIMD on 256 CUs: the issue pattern that sustains the most
    n = waves * 16 * 64 * 8        # bf16 operand elements
    sink = torch.empty(waves * 64, dtype=torch.float32, device="cuda")
    gen = torch.Generator(device="cuda")
    gen.manual_seed(2606200050 + 9)
    out = {"kernel": "v_mfma_f32_32x32x16_bf16, 4 independent accumulators, 1 wave per SIMD",
           "waves": waves, "iters": iters}
    flop = waves * iters * 16 * 32768
    stream = torch.cuda.current_stream()
    for label, src in (("randn", torch.randn(n, generator=gen, device="cuda").to(torch.bfloat16)),
                       ("ones", torch.ones(n, dtype=torch.bfloat16, device="cuda"))):
        def call():
            st = lib.streamkl_bench_mfma_peak(ctypes.c_void_p(src.data_ptr()), waves, iters,
                                              ctypes.c_void_p(sink.data_ptr()), ctypes.c_void_p(stream.cuda_stream))
            assert st == 0, st
        call()
        torch.cuda.synchronize()
        ms = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            call()
            e1.record(stream)
            torch.cuda.synchronize()
            ms.append(e0.elapsed_time(e1))
        med = statistics.median(ms)
        out[f"tflops_{label}"] = round(flop / (med * 1e-3) / 1e12, 1)
        out[f"frac_bf16_peak_{label}"] = round(flop / (med * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)
        del src
    torch.cuda.empty_cache()
    return out


def timed_reps(fn, reps, evict=None):
    """Median and min of `reps` event-timed calls of fn (each after evict() when given)."""
    import torch
    fn()
    torch.cuda.synchronize()
    ms = []
    for _ in range(reps):
        if evict is not None:
            evict()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        fn()
        e1.record()
        torch.cuda.synchronize()
        ms.append(e0.elapsed_time(e1))
    return statistics.median(ms), min(ms)


def split_k_figures(sk, evict, reps=10):
    """Split-K forward (Sec. 3.3) against the single pass on decode-like shapes:
    16 heads of N_Q in {1, 16, 32, 64} rows over N_K = 65536 keys, d1 = d2 = 128,
    non-causal (the shape family of the paper's split-K ablation). Inputs are
    seeded N(0,1) drawn on the device; median of `reps` event-timed calls,
    each after a cache eviction (Evictor)."""
    import torch
    B, H, NK, D = 16, 1, 65536, 128
    gen = torch.Generator(device="cuda")
    gen.manual_seed(2606200050 + 6)
    k1 = torch.randn((B, H, NK, D), generator=gen, device="cuda").to(torch.bfloat16)
    k2 = torch.randn((B, H, NK, D), generator=gen, device="cuda").to(torch.bfloat16)
    s = D ** -0.5
    out = []
    for nq in (1, 16, 32, 64):
        q1 = torch.randn((B, H, nq, D), generator=gen, device="cuda").to(torch.bfloat16)
        q2 = torch.randn((B, H, nq, D), generator=gen, device="cuda").to(torch.bfloat16)
        res = {"n_q": nq}
        for label, fn in (("single_pass", lambda: sk.fwd(q1, k1, q2, k2, s, s, False, 0)),
                          ("split", lambda: sk.fwd_split(q1, k1, q2, k2, s, s, False, 0, splits="auto"))):
            med, _ = timed_reps(fn, reps, evict)
            res[label + "_ms"] = round(med, 4)
        res["splits"] = sk.split_count(B, H, nq, NK, D, D)
        res["speedup"] = round(res["single_pass_ms"] / res["split_ms"], 2)
        res["split_tflops"] = round(2 * 2 * D * B * H * nq * NK / (res["split_ms"] * 1e-3) / 1e12, 2)
        res["split_k_stream_tbps"] = round(2 * D * 2 * B * H * NK / (res["split_ms"] * 1e-3) / 1e12, 2)
        out.append(res)
    del k1, k2
    torch.cuda.empty_cache()
    return {"workload": f"B={B} H={H} N_K={NK} d1=d2={D} non-causal, N_Q in (1, 16, 32, 64)", "rows": out}


def clock_figures(sk, reps=10):
    """The mid forward (32 heads, 16384 x 16384, d = 128, non-causal) and a
    library bf16 GEMM (torch.matmul, 8192^3) on seeded N(0,1) operands and on
    constant operands of the same shapes: identical instruction streams, so a
    difference in time is a difference in clock. The shader clock itself is
    read under rocprofv3 --pmc GRBM_GUI_ACTIVE (cycles per dispatch, summed
    over the eight XCDs, divided by the dispatch's duration)."""
    import torch
    w = {"B": 1, "H": 32, "n": 16384, "d": 128}
    shape = (w["B"], w["H"], w["n"], w["d"])
    s = w["d"] ** -0.5
    gen = torch.Generator(device="cuda")
    gen.manual_seed(2606200050 + 8)
    out = {"workload": "forward: B=1 H=32 N_Q=N_K=16384 d1=d2=128 non-causal; GEMM: bf16 8192 x 8192 x 8192 "
                       "(torch.matmul, reference only)"}
    fwd_flop = 2 * 2 * w["d"] * w["B"] * w["H"] * w["n"] * w["n"]
    gemm_n = 8192
    for label, make in (("randn", lambda sh: torch.randn(sh, generator=gen, device="cuda").to(torch.bfloat16)),
                        ("ones", lambda sh: torch.ones(sh, device="cuda", dtype=torch.bfloat16))):
        q1, k1, q2, k2 = (make(shape) for _ in range(4))
        ms, _ = timed_reps(lambda: sk.fwd(q1, k1, q2, k2, s, s, False, 0), reps)
        out[f"fwd_ms_{label}"] = round(ms, 4)
        out[f"fwd_tflops_{label}"] = round(fwd_flop / (ms * 1e-3) / 1e12, 2)
        del q1, k1, q2, k2
        a, b = make((gemm_n, gemm_n)), make((gemm_n, gemm_n))
        ms, _ = timed_reps(lambda: torch.matmul(a, b), reps)
        out[f"gemm_tflops_{label}"] = round(2 * gemm_n ** 3 / (ms * 1e-3) / 1e12, 2)
        del a, b
    torch.cuda.empty_cache()
    return out


def fused_bwd_figures(sk, evict, reps=10):
    """Backward strategies of Sec. 4.2 on the same decode-like shapes as the
    split-K figures (16 heads, N_K = 65536, d1 = d2 = 128, non-causal, student
    gradients dQ2 and dK2), plus 512 query rows near the measured crossover:
    the separate dQ/dK kernels against the fused key-owned kernel with atomic
    dQ, and the strategy the adaptive rule picks. Median of `reps` calls each,
    after a cache eviction (Evictor)."""
    import torch
    B, H, NK, D = 16, 1, 65536, 128
    gen = torch.Generator(device="cuda")
    gen.manual_seed(2606200050 + 7)
    mk = lambda n: torch.randn((B, H, n, D), generator=gen, device="cuda").to(torch.bfloat16)  # noqa: E731
    k1, k2 = mk(NK), mk(NK)
    s = D ** -0.5
    out = []
    for nq in (1, 16, 32, 64, 512):
        q1, q2 = mk(nq), mk(nq)
        kl, l1, l2 = sk.fwd(q1, k1, q2, k2, s, s, False, 0)
        g = torch.full((B, H, nq), 1.0 / (B * H * nq), device="cuda")
        grads = {"dq2": torch.empty((B, H, nq, D), device="cuda"), "dk2": torch.empty((B, H, NK, D), device="cuda")}
        res = {"n_q": nq}
        for strat in ("separate", "fused"):
            fn = lambda: sk.bwd(q1, k1, q2, k2, kl, l1, l2, g, s, s, False, 0, out=grads, strategy=strat)  # noqa: E731
            med, _ = timed_reps(fn, reps, evict)
            res[strat + "_ms"] = round(med, 4)
        res["speedup"] = round(res["separate_ms"] / res["fused_ms"], 2)
        res["auto_picks"] = sk.bwd_choose(B, H, nq, NK, D, D)
        # compulsory bytes of the fused pass: K1, K2 read once, dK2 written, dQ2 added
        byts = B * H * (2 * NK * D * 2 + NK * D * 4 + 2 * nq * D * 2 + nq * D * 4)
        res["fused_hbm_tbps"] = round(byts / (res["fused_ms"] * 1e-3) / 1e12, 2)
        out.append(res)
        del q1, q2, kl, l1, l2, g, grads
    del k1, k2
    torch.cuda.empty_cache()
    return {"workload": f"B={B} H={H} N_K={NK} d1=d2={D} non-causal, dQ2 + dK2, N_Q in (1, 16, 32, 64, 512)",
            "rows": out}


def sigmoid_figures(sk, evict, reps=10):
    """The sigmoid-score path (streamkl_fwd_act / streamkl_bwd_act, Sec. 3.1)
    on the mid shape (32 heads, 16384 x 16384, d1 = d2 = 128, seeded N(0,1)
    drawn on the device), non-causal and causal: forward, dQ2 and dK2 kernels,
    median of `reps` event-timed calls each after a cache eviction (Evictor).
    TFLOP/s count the same MFMA work as the softmax path; the kernels
    themselves are bound by vector and transcendental issue (per score
    pair: two v_exp_f32 and two v_rcp_f32, and one v_log_f32 where the
    log-ratio is needed)."""
    import torch
    B, H, N, D = 1, 32, 16384, 128
    gen = torch.Generator(device="cuda")
    gen.manual_seed(2606200050 + 10)
    q1, k1, q2, k2 = (torch.randn((B, H, N, D), generator=gen, device="cuda").to(torch.bfloat16) for _ in range(4))
    s = D ** -0.5
    g = torch.full((B, H, N), 1.0 / (B * H * N), device="cuda")
    dq2, dk2 = torch.empty((B, H, N, D), device="cuda"), torch.empty((B, H, N, D), device="cuda")
    out = []
    f = flops_per_pair(D, D)
    for causal in (False, True):
        P = B * H * (N * (N + 1) // 2 if causal else N * N)
        fns = {"fwd": lambda: sk.fwd_act(q1, k1, q2, k2, s, s, causal, 0, "sigmoid"),
               "dq": lambda: sk.bwd(q1, k1, q2, k2, None, None, None, g, s, s, causal, 0, want=("dq2",),
                                    out={"dq2": dq2}, activation="sigmoid"),
               "dk": lambda: sk.bwd(q1, k1, q2, k2, None, None, None, g, s, s, causal, 0, want=("dk2",),
                                    out={"dk2": dk2}, activation="sigmoid")}
        row = {"causal": causal, "pairs": P}
        for k, fn in fns.items():
            med, _ = timed_reps(fn, reps, evict)
            row[f"{k}_ms"] = round(med, 4)
            row[f"{k}_tflops"] = round(f[k] * P / (med * 1e-3) / 1e12, 2)
        row["bwd_tflops_algorithmic"] = round(f["bwd"] * P / ((row["dq_ms"] + row["dk_ms"]) * 1e-3) / 1e12, 2)
        out.append(row)
    del q1, k1, q2, k2, dq2, dk2
    torch.cuda.empty_cache()
    return {"workload": f"sigmoid scores, generalized KL: B={B} H={H} N_Q=N_K={N} d1=d2={D}", "rows": out}


# ---------------------------------------------------------------------------- CPU baseline (the fp64 oracle)

_CPU = {}


def _cpu_worker_init(arrays, w):
    from threadpoolctl import threadpool_limits
    threadpool_limits(1)        # one BLAS thread per worker process
    _CPU["a"] = arrays
    _CPU["w"] = w


def _cpu_worker(job):
    """Row blocks of one head (all keys each) until `budget` seconds pass; returns (rows, seconds)."""
    import numpy as np
    import oracle
    h, budget, with_bwd = job
    w = _CPU["w"]
    Q1, K1, Q2, K2 = (_CPU["a"][k][:, h:h + 1] for k in ("Q1", "K1", "Q2", "K2"))
    block, r0, rows = 128, 0, 0
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < budget:
        r = slice(r0 % w.n_q, r0 % w.n_q + block)
        if with_bwd:
            oracle.backward(Q1[:, :, r], K1, Q2[:, :, r], K2, w.s1, w.s2, False, 0, np.ones((1, 1, block)),
                            row_block=block)
        else:
            oracle.forward(Q1[:, :, r], K1, Q2[:, :, r], K2, w.s1, w.s2, False, 0, row_block=block)
        r0 += block
        rows += block
    return rows, time.perf_counter() - t0


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(w, budget_fwd=6.0, budget_bwd=10.0, max_workers=16):
    """The fp64 oracle as it stands, on a bounded sample of the workload: one worker process per head
    (heads 0, 1, ...), each forward-only for budget_fwd seconds and then forward + student backward for
    budget_bwd seconds over its head's query rows in blocks of 128, all keys each (non-causal)."""
    import multiprocessing as mp
    from paper_2606_20005_amd import inputs
    n_cpu = os.cpu_count() or 1
    workers = max(1, min(n_cpu, max_workers, w.H))
    small = inputs.make(w, H=workers)          # the first heads of the workload's seeded tensors
    arrays = {k: small[k] for k in ("Q1", "K1", "Q2", "K2")}
    f = flops_per_pair(w.d1, w.d2)
    res = {"unit": "TFLOP/s", "kind": "oracle", "cores": workers, "os_cpu_count": n_cpu, "cpu_model": _cpu_model()}
    ctx = mp.get_context("spawn")
    with ctx.Pool(workers, initializer=_cpu_worker_init, initargs=(arrays, w)) as pool:
        for label, budget, with_bwd, fpp in (("fwd", budget_fwd, False, f["fwd"]),
                                              ("fwd_bwd", budget_bwd, True, f["fwd"] + f["bwd"])):
            t0 = time.perf_counter()
            out = pool.map(_cpu_worker, [(h, budget, with_bwd) for h in range(workers)])
            wall = time.perf_counter() - t0
            rows = sum(r for r, _ in out)
            P = rows * w.n_k
            res[f"{label}_tflops"] = round(fpp * P / wall / 1e12, 6)
            res[f"{label}_rows"] = rows
            res[f"{label}_seconds"] = round(wall, 2)
    res["value"] = res["fwd_bwd_tflops"]
    res["sample"] = (f"{workers} worker processes (one BLAS thread each), worker h on head h of the mid workload: "
                     f"query rows in blocks of 128 x all {w.n_k} keys (non-causal) in fp64 numpy, "
                     f"{budget_fwd:.0f} s forward only ({res['fwd_rows']} rows), then {budget_bwd:.0f} s forward + "
                     f"student backward ({res['fwd_bwd_rows']} rows); value = the latter, algorithmic TFLOP/s")
    return res


# ---------------------------------------------------------------------------- main

def roofline_obj(name, flop, ms, traffic=None):
    tf = flop / (ms * 1e-3) / 1e12
    return {"kernel": name, "bound": "mfma", "achieved": round(tf, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
            "frac": round(tf / PEAK_BF16_TFLOPS, 4), "traffic": traffic, "flop_per_launch": flop,
            "avg_launch_ms": round(ms, 4)}


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--reps", type=int, default=20, help="cache-evicted event-timed steps per workload (>= 10 at 64K)")
    ap.add_argument("--no-64k", action="store_true", help="skip the 64K long-context figures")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-split", action="store_true", help="skip the split-K decode-shape figures")
    ap.add_argument("--no-fused", action="store_true", help="skip the fused-backward decode-shape figures")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the per-pass figures of the other workloads (distill, mid causal, indexer)")
    ap.add_argument("--causal", action="store_true", help="run the 16K workload with causal masking")
    ap.add_argument("--no-clock-probe", action="store_true",
                    help="skip timing the mid forward and a library GEMM on random and on constant operands")
    ap.add_argument("--no-mfma-peak", action="store_true", help="skip the measured MFMA peak")
    ap.add_argument("--no-sigmoid", action="store_true", help="skip the sigmoid-score figures")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after timing, run one 1 GiB device copy (reference kernel for HBM counters)")
    a = ap.parse_args()
    if a.gpus != 1:
        print(f"bench.py runs on exactly one GPU (asked for {a.gpus}): the attention-KL path has no "
              "multi-GPU code; B*H shards across GPUs without communication", file=sys.stderr)
        return 2

    from paper_2606_20005_amd import inputs
    w = inputs.WORKLOADS["mid"]
    cpu = None
    if not a.no_cpu_baseline:          # before anything touches the GPU: its workers are spawned processes
        cpu = cpu_baseline(w)

    import torch
    from paper_2606_20005_amd import streamkl as sk
    if not torch.cuda.is_available():
        print("bench.py needs an MI355X GPU", file=sys.stderr)
        return 2
    evict = Evictor()
    peak = None if a.no_mfma_peak else mfma_peak_figures()
    peak_meas = peak["tflops_randn"] if peak else None
    causal = bool(a.causal)
    wall_ms, times, extra, kl_mean = run_workload(sk, w, causal, a.steps, a.warmup, a.reps, evict)
    kern, P, f = summarize(w, causal, times, peak_meas)
    step_flop = (f["fwd"] + f["bwd"]) * P
    value = step_flop / (wall_ms * 1e-3) / 1e12
    dom = max(("fwd", "dq", "dk"), key=lambda k: kern[k]["ms_median"])
    roof = roofline_obj(KERNEL_NAMES[dom], kern[dom]["flop_per_launch"], kern[dom]["ms_median"],
                        measured_traffic(KERNEL_NAMES[dom]))
    roof["accounting"] = ("algorithmic flop per launch: forward 2(d1+d2) per pair; each separate backward kernel "
                          "its contraction 2 d2 plus half the recompute (d1+d2) per pair")
    res = {
        "metric": "fused attn-KL fwd/bwd TFLOP/s + ms at N=16K/64K; % bf16 MFMA peak; extra HBM",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(wall_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1), bf16-rounded; Q2 = Q1 + 0.3 eps, K2 = K1)",
        "config": {"workload": "mid: B=1 H=32 N_Q=N_K=16384 d1=d2=128 " + ("causal" if causal else "non-causal")
                   + ", fwd + bwd(dQ2, dK2), mean objective", "B": w.B, "H": w.H, "n_q": w.n_q, "n_k": w.n_k,
                   "d1": w.d1, "d2": w.d2, "causal": causal, "pairs": P},
        "passes": {"fwd_ms": kern["fwd"]["ms_median"], "fwd_tflops": kern["fwd"]["tflops"],
                   "fwd_frac_bf16_peak": kern["fwd"]["frac_bf16_peak"],
                   "bwd_ms": kern["bwd"]["ms_median"], "bwd_tflops_algorithmic": kern["bwd"]["tflops"],
                   "bwd_frac_bf16_peak": kern["bwd"]["frac_bf16_peak"],
                   "event_step_ms": round(kern["fwd"]["ms_median"] + kern["bwd"]["ms_median"], 4),
                   "timing": f"median of {a.reps} steps, each after a {EVICT_BYTES >> 20} MiB write and a {EVICT_BYTES >> 20} MiB read that leave the MALL without the workload's data or dirty lines"},
        "kernels": {k: kern[k] for k in ("fwd", "dq", "dk")},
        "roofline": roof,
        "roofline_target": roofline_obj(KERNEL_NAMES["fwd"], kern["fwd"]["flop_per_launch"], kern["fwd"]["ms_median"],
                                        measured_traffic(KERNEL_NAMES["fwd"])),
        "roofline_bwd_pass": roofline_obj(KERNEL_NAMES["dq"] + " + " + KERNEL_NAMES["dk"], kern["bwd"]["flop"],
                                          kern["bwd"]["ms_median"]),
        "extra_hbm": extra,
        "kl_mean": kl_mean,
    }
    if peak:
        res["mfma_peak"] = peak
        for r in ("roofline", "roofline_target", "roofline_bwd_pass"):
            res[r]["frac_measured_peak"] = round(res[r]["achieved"] / peak_meas, 4)
    if not a.no_64k:
        wl = inputs.WORKLOADS["long"]
        wall_l, times_l, extra_l, kl_l = run_workload(sk, wl, True, 3, 2, max(10, min(a.reps, 10)), evict)
        kern_l, P_l, f_l = summarize(wl, True, times_l, peak_meas)
        res["long_context"] = {
            "workload": "long: B=1 H=32 N_Q=N_K=65536 d1=128 d2=64 causal, outlier channels",
            "pairs": P_l, "ms_per_step": round(wall_l, 4),
            **{k: kern_l[k] for k in ("fwd", "dq", "dk", "bwd")},
            "extra_hbm": extra_l, "extra_hbm_o_nq_bytes": extra_l["workspace_bytes"] + extra_l["stats_bytes"],
            "naive_p1_p2_bytes": 2 * 2 * P_l, "kl_mean": kl_l}
    if not a.no_workloads:
        rows = []
        for name, wc in (("distill", True), ("mid", True), ("indexer", True)):
            wo = inputs.WORKLOADS[name]
            wall_o, times_o, _, kl_o = run_workload(sk, wo, wc, 3, 2, 10, evict)
            kern_o, P_o, f_o = summarize(wo, wc, times_o, peak_meas)
            rows.append({"workload": f"{name}: B={wo.B} H={wo.H} N_Q={wo.n_q} N_K={wo.n_k} d1={wo.d1} d2={wo.d2} "
                                     + ("causal" if wc else "non-causal"),
                         "pairs": P_o, "ms_per_step": round(wall_o, 4),
                         **{f"{k}_ms": kern_o[k]["ms_median"] for k in ("fwd", "dq", "dk")},
                         **{f"{k}_frac_bf16_peak": kern_o[k]["frac_bf16_peak"] for k in ("fwd", "dq", "dk", "bwd")},
                         "step_tflops_algorithmic": round(
                             (f_o["fwd"] + f_o["bwd"]) * P_o / (wall_o * 1e-3) / 1e12, 2),
                         "kl_mean": kl_o})
        res["workloads"] = rows
    if not a.no_split:
        res["split_k"] = split_k_figures(sk, evict)
    if not a.no_fused:
        res["fused_bwd"] = fused_bwd_figures(sk, evict)
    if not a.no_sigmoid:
        res["sigmoid"] = sigmoid_figures(sk, evict)
    if not a.no_clock_probe:
        res["clock_probe"] = clock_figures(sk)
    if a.copy_calibration:
        x = torch.empty(1 << 28, dtype=torch.float32, device="cuda")   # 1 GiB
        y = torch.empty_like(x)
        torch.cuda.synchronize()
        y.copy_(x)
        torch.cuda.synchronize()
        res["copy_calibration_bytes"] = {"read": x.numel() * 4, "write": y.numel() * 4}
        del x, y
    if cpu is not None:
        res["cpu_baseline"] = cpu
    print(json.dumps(res), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
