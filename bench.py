#!/usr/bin/env python3
"""Throughput of the fused attention-distillation KL on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input:
the forward (streamkl_fwd: KL, LSE1, LSE2 for every row) followed by the
standard-distillation backward (streamkl_bwd: dQ2 via the query-owned kernel,
then dK2 via the key-owned kernel) with the paper's mean objective
(dkl = 1 / (B H N_Q)). Inputs are resident in HBM before timing starts.

Workload (the one the 16K figure is quoted on): B=1, H=32, N_Q=N_K=16384,
d1=d2=128, s=1/sqrt(128), non-causal, student Q2 = bf16(Q1 + 0.3 eps), K2 = K1.
Prints ONE JSON line. The 64K causal long-context figures (d1=128, d2=64,
outlier channels) ride along in "long_context" unless --no-64k, and the
split-K forward on decode-like shapes (16 heads of 1-64 query rows over 64K
keys) in "split_k" unless --no-split, the separate against the fused
backward on the same shapes in "fused_bwd" unless --no-fused, and the
per-pass figures of the other causal workloads (distill, mid, indexer) in
"workloads" unless --no-workloads.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-64k] [--no-cpu-baseline] [--no-split] [--no-fused]
                    [--no-workloads]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBPS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.json")


def kernel_source_hash():
    """SHA-256 over the code of the HIP sources and the C header: counters are only valid for the code they
    measured. Comments and layout are left out, so editing a comment keeps the measurement."""
    import glob
    import hashlib
    import re
    h = hashlib.sha256()
    files = sorted(glob.glob(os.path.join(ROOT, "paper_2606_20005_amd", "csrc", "*"))) + \
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


def flops_per_pair(w):
    d1, d2 = w.d1, w.d2
    return {
        "fwd": 2 * (d1 + d2),                 # S1 and S2
        "dq": 2 * (d1 + d2) + 2 * d2,         # recompute S1, S2; dQ2 = dS2 K2
        "dk": 2 * (d1 + d2) + 2 * d2,         # recompute S1, S2; dK2 = dS2^T Q2
        "bwd_algorithmic": 2 * (d1 + d2) + 4 * d2,   # recompute counted once (fused ideal)
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


def run_workload(sk, w, causal, steps, warmup):
    """Time `steps` steps; returns per-kernel mean ms (HIP events on the launch stream) and wall ms/step."""
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
        sk.bwd(q1, k1, q2, k2, kl, l1, l2, g, w.s1, w.s2, causal, 0, want=("dq2",), out={"dq2": dq2})
        if ev is not None:
            ev[2].record(stream)
        sk.bwd(q1, k1, q2, k2, kl, l1, l2, g, w.s1, w.s2, causal, 0, want=("dk2",), out={"dk2": dk2})
        if ev is not None:
            ev[3].record(stream)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    free0, total_mem = torch.cuda.mem_get_info()
    alloc0 = torch.cuda.max_memory_allocated()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(steps):
        step(events[s])
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3 / steps
    free1, _ = torch.cuda.mem_get_info()
    ms = {"fwd": 0.0, "dq": 0.0, "dk": 0.0}
    for ev in events:
        ms["fwd"] += ev[0].elapsed_time(ev[1]) / steps
        ms["dq"] += ev[1].elapsed_time(ev[2]) / steps
        ms["dk"] += ev[2].elapsed_time(ev[3]) / steps
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
    return ms, wall_ms, extra, kl_mean


def split_k_figures(sk, reps=10):
    """Split-K forward (Sec. 3.3) against the single pass on decode-like shapes:
    16 heads of N_Q in {1, 16, 32, 64} rows over N_K = 65536 keys, d1 = d2 = 128,
    non-causal (the shape family of the paper's split-K ablation). Inputs are
    seeded N(0,1) drawn on the device; HIP events over `reps` launches each."""
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
            fn()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                fn()
            e1.record()
            torch.cuda.synchronize()
            res[label + "_ms"] = round(e0.elapsed_time(e1) / reps, 4)
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

    out = {"workload": "forward: B=1 H=32 N_Q=N_K=16384 d1=d2=128 non-causal; GEMM: bf16 8192 x 8192 x 8192 "
                       "(torch.matmul, reference only)"}
    fwd_flop = 2 * 2 * w["d"] * w["B"] * w["H"] * w["n"] * w["n"]
    gemm_n = 8192
    for label, make in (("randn", lambda sh: torch.randn(sh, generator=gen, device="cuda").to(torch.bfloat16)),
                        ("ones", lambda sh: torch.ones(sh, device="cuda", dtype=torch.bfloat16))):
        q1, k1, q2, k2 = (make(shape) for _ in range(4))
        ms = timed(lambda: sk.fwd(q1, k1, q2, k2, s, s, False, 0))
        out[f"fwd_ms_{label}"] = round(ms, 4)
        out[f"fwd_tflops_{label}"] = round(fwd_flop / (ms * 1e-3) / 1e12, 2)
        del q1, k1, q2, k2
        a, b = make((gemm_n, gemm_n)), make((gemm_n, gemm_n))
        ms = timed(lambda: torch.matmul(a, b))
        out[f"gemm_tflops_{label}"] = round(2 * gemm_n ** 3 / (ms * 1e-3) / 1e12, 2)
        del a, b
    torch.cuda.empty_cache()
    return out


def fused_bwd_figures(sk, reps=10):
    """Backward strategies of Sec. 4.2 on the same decode-like shapes as the
    split-K figures (16 heads, N_K = 65536, d1 = d2 = 128, non-causal, student
    gradients dQ2 and dK2), plus 512 query rows near the measured crossover:
    the separate dQ/dK kernels against the fused key-owned kernel with atomic
    dQ, and the strategy the adaptive rule picks. HIP events over `reps`
    calls each."""
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
            fn()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                fn()
            e1.record()
            torch.cuda.synchronize()
            res[strat + "_ms"] = round(e0.elapsed_time(e1) / reps, 4)
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


def summarize(w, causal, ms):
    P = pairs(w, causal)
    f = flops_per_pair(w)
    out = {}
    for k in ("fwd", "dq", "dk"):
        tf = f[k] * P / (ms[k] * 1e-3) / 1e12
        out[k] = {"ms": round(ms[k], 4), "tflops": round(tf, 2), "frac_bf16_peak": round(tf / PEAK_BF16_TFLOPS, 4),
                  "flop_per_launch": f[k] * P}
    bwd_ms = ms["dq"] + ms["dk"]
    out["bwd"] = {"ms": round(bwd_ms, 4),
                  "tflops_algorithmic": round(f["bwd_algorithmic"] * P / (bwd_ms * 1e-3) / 1e12, 2)}
    return out, P, f


def cpu_baseline(w, budget_s=15.0, max_heads=2):
    """The fp64 oracle on a bounded sample: row blocks of heads 0, 1, ... (all keys each), fwd + student bwd,
    until about budget_s seconds of CPU work."""
    import numpy as np
    import oracle
    from paper_2606_20005_amd import inputs
    small = inputs.make(w, H=max_heads)   # the first heads of the workload's seeded tensors
    rows_done = 0
    block = 128
    t0 = time.perf_counter()
    for h in range(max_heads):
        Q1, K1, Q2, K2 = (small[k][:, h:h + 1] for k in ("Q1", "K1", "Q2", "K2"))
        r0 = 0
        while r0 < w.n_q and time.perf_counter() - t0 < budget_s:
            r = slice(r0, min(w.n_q, r0 + block))
            oracle.backward(Q1[:, :, r], K1, Q2[:, :, r], K2, w.s1, w.s2, False, 0,
                            np.ones((1, 1, r.stop - r.start)), row_block=block)
            r0 = r.stop
            rows_done += r.stop - r.start
    dt = time.perf_counter() - t0
    f = flops_per_pair(w)
    P = rows_done * w.n_k
    tflops = (f["fwd"] + f["bwd_algorithmic"]) * P / dt / 1e12
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:   # pragma: no cover
        cores = 1
    return {"value": round(tflops, 6), "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
            "sample": f"{rows_done} query rows (head 0 first, then head 1) x all {w.n_k} keys (non-causal), "
                      f"forward + student backward in fp64 (numpy), {dt:.1f} s",
            "seconds": round(dt, 2), "pairs": P}


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-64k", action="store_true", help="skip the 64K long-context figures")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-split", action="store_true", help="skip the split-K decode-shape figures")
    ap.add_argument("--no-fused", action="store_true", help="skip the fused-backward decode-shape figures")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the per-pass figures of the other workloads (distill, mid causal, indexer)")
    ap.add_argument("--causal", action="store_true", help="run the 16K workload with causal masking")
    ap.add_argument("--no-clock-probe", action="store_true",
                    help="skip timing the mid forward and a library GEMM on random and on constant operands")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after timing, run one 1 GiB device copy (reference kernel for HBM counters)")
    a = ap.parse_args()
    if a.gpus != 1:
        print(f"bench.py runs on exactly one GPU (asked for {a.gpus}): the attention-KL path has no "
              "multi-GPU code; B*H shards across GPUs without communication", file=sys.stderr)
        return 2

    import torch
    from paper_2606_20005_amd import inputs, streamkl as sk
    if not torch.cuda.is_available():
        print("bench.py needs an MI355X GPU", file=sys.stderr)
        return 2
    w = inputs.WORKLOADS["mid"]
    causal = bool(a.causal)
    ms, wall_ms, extra, kl_mean = run_workload(sk, w, causal, a.steps, a.warmup)
    kern, P, f = summarize(w, causal, ms)
    step_ms = ms["fwd"] + ms["dq"] + ms["dk"]
    step_flop = (f["fwd"] + f["bwd_algorithmic"]) * P
    value = step_flop / (wall_ms * 1e-3) / 1e12
    dom = max(("fwd", "dq", "dk"), key=lambda k: ms[k])
    names = {"fwd": "kl_fwd_kernel<128,128>", "dq": "kl_bwd_dq_kernel<128,128,mode1>",
             "dk": "kl_bwd_dk_kernel<128,128,mode1>"}
    achieved = kern[dom]["tflops"]
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
        "passes": {"fwd_ms": kern["fwd"]["ms"], "fwd_tflops": kern["fwd"]["tflops"],
                   "fwd_frac_bf16_peak": kern["fwd"]["frac_bf16_peak"],
                   "bwd_ms": kern["bwd"]["ms"], "bwd_tflops_algorithmic": kern["bwd"]["tflops_algorithmic"],
                   "bwd_frac_bf16_peak": round(kern["bwd"]["tflops_algorithmic"] / PEAK_BF16_TFLOPS, 4),
                   "event_step_ms": round(step_ms, 4)},
        "kernels": {k: kern[k] for k in ("fwd", "dq", "dk")},
        "roofline": {"kernel": names[dom], "bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": measured_traffic(names[dom]),
                     "flop_per_launch": kern[dom]["flop_per_launch"], "avg_launch_ms": kern[dom]["ms"]},
        "extra_hbm": extra,
        "kl_mean": kl_mean,
    }
    if not a.no_64k:
        wl = inputs.WORKLOADS["long"]
        ms_l, wall_l, extra_l, kl_l = run_workload(sk, wl, True, max(2, min(a.steps, 3)), 1)
        kern_l, P_l, f_l = summarize(wl, True, ms_l)
        res["long_context"] = {
            "workload": "long: B=1 H=32 N_Q=N_K=65536 d1=128 d2=64 causal, outlier channels",
            "pairs": P_l, "fwd_ms": kern_l["fwd"]["ms"], "fwd_tflops": kern_l["fwd"]["tflops"],
            "fwd_frac_bf16_peak": kern_l["fwd"]["frac_bf16_peak"], "bwd_ms": kern_l["bwd"]["ms"],
            "bwd_tflops_algorithmic": kern_l["bwd"]["tflops_algorithmic"],
            "dq_ms": kern_l["dq"]["ms"], "dq_tflops": kern_l["dq"]["tflops"],
            "dk_ms": kern_l["dk"]["ms"], "dk_tflops": kern_l["dk"]["tflops"], "extra_hbm": extra_l,
            "naive_p1_p2_bytes": 2 * 2 * P_l, "kl_mean": kl_l}
    if not a.no_workloads:
        rows = []
        for name, wc in (("distill", True), ("mid", True), ("indexer", True)):
            wo = inputs.WORKLOADS[name]
            ms_o, wall_o, _, kl_o = run_workload(sk, wo, wc, 3, 1)
            kern_o, P_o, f_o = summarize(wo, wc, ms_o)
            rows.append({"workload": f"{name}: B={wo.B} H={wo.H} N_Q={wo.n_q} N_K={wo.n_k} d1={wo.d1} d2={wo.d2} "
                                     + ("causal" if wc else "non-causal"),
                         "pairs": P_o, "ms_per_step": round(wall_o, 4),
                         **{f"{k}_ms": kern_o[k]["ms"] for k in ("fwd", "dq", "dk")},
                         **{f"{k}_frac_bf16_peak": kern_o[k]["frac_bf16_peak"] for k in ("fwd", "dq", "dk")},
                         "step_tflops_algorithmic": round(
                             (f_o["fwd"] + f_o["bwd_algorithmic"]) * P_o / (wall_o * 1e-3) / 1e12, 2),
                         "kl_mean": kl_o})
        res["workloads"] = rows
    if not a.no_split:
        res["split_k"] = split_k_figures(sk)
    if not a.no_fused:
        res["fused_bwd"] = fused_bwd_figures(sk)
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
    if not a.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(res), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
