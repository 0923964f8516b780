"""GPU parity at the full workload sizes, in the configuration the benchmark
launches (student gradients dQ2, dK2 of KL(P1 || P2)).

The oracle cannot evaluate a whole 16K-128K head in seconds, so each workload
is checked on sampled outputs that it computes one by one:
  * KL, LSE1, LSE2 and dQ2 of sampled query rows (first, last, tile edges and
    random rows) of three heads;
  * dK2 of sampled keys of one head (random keys where the oracle can afford
    the head's full statistics, else the last keys, which under the causal
    mask only the last rows attend);
and on properties that hold at any size, over every row and head:
  * KL >= 0 (Gibbs) within the row tolerance, LSE finite;
  * sum_j dK2[j] = 0 (each row of dS sums to zero);
  * <dQ2, Q2> = <dK2, K2> per head (both equal sum_ij dS_ij S_ij).
The property tolerances are relative to the magnitude of the summed terms: dS
is rounded to bf16 before the second product, which breaks the exact zero
row sums by at most 2^-9 per term.
"""
import time

import numpy as np
import pytest

import oracle
from paper_2606_20005_amd import inputs
from parity_utils import GRAD_REL_L2, KL_ATOL, check_grad, check_rows, to_gpu_f32, upload

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

PROPERTY_REL = 1e-2


def _sample_rows(n_q, rng, k=48):
    fixed = [0, 1, 31, 32, 127, 128, n_q // 2, n_q - 129, n_q - 128, n_q - 2, n_q - 1]
    extra = rng.choice(n_q, size=k, replace=False)
    return np.unique(np.clip(np.concatenate([fixed, extra]), 0, n_q - 1))


def _sample_keys(w, causal, rng, full_stats_ok, k=24):
    if full_stats_ok or not causal:
        fixed = [0, 1, 127, 128, w.n_k // 2, w.n_k - 1]
        extra = rng.choice(w.n_k, size=k, replace=False)
    else:
        lo = w.n_k - 1024   # rows attending these keys: the last 1024 + (N_Q - N_K) ones
        fixed = [lo, lo + 127, lo + 128, w.n_k - 129, w.n_k - 128, w.n_k - 1]
        extra = lo + rng.choice(1024, size=k, replace=False)
    return np.unique(np.concatenate([fixed, extra]))


def _log(msg):
    print(msg, flush=True)


def _run_full(sk, name, causal, full_stats_ok):
    import torch
    t0 = time.time()
    d = inputs.make(name)
    w = d["w"]
    _log(f"[fullsize] {name} causal={causal} B={w.B} H={w.H} NQ={w.n_q} NK={w.n_k} d1={w.d1} d2={w.d2}")
    q1, k1, q2, k2 = upload(d)
    g = to_gpu_f32(d["g"])
    kl, l1, l2 = sk.fwd(q1, k1, q2, k2, w.s1, w.s2, causal, 0)
    _, _, dq2, dk2 = sk.bwd(q1, k1, q2, k2, kl, l1, l2, g, w.s1, w.s2, causal, 0, want=("dq2", "dk2"))
    torch.cuda.synchronize()
    _log(f"[fullsize] {name}: inputs + GPU pass {time.time() - t0:.1f} s")

    # --- properties over every row and head
    assert bool(torch.isfinite(kl).all()) and bool(torch.isfinite(l1).all()) and bool(torch.isfinite(l2).all())
    assert float(kl.min()) >= -KL_ATOL, f"KL below zero: {float(kl.min())}"
    assert bool(torch.isfinite(dq2).all()) and bool(torch.isfinite(dk2).all())
    dq = dq2.double()
    dk = dk2.double()
    q2d = q2.double()
    k2d = k2.double()
    col_sum = dk.sum(dim=2)                                     # [B, H, d2]
    dk_norm = dk.pow(2).sum(dim=(2, 3)).sqrt()                  # [B, H]
    ratio = (col_sum.pow(2).sum(dim=2).sqrt() / dk_norm).max().item()
    _log(f"[fullsize] {name}: max_h ||sum_j dK2[j]|| / ||dK2||_F = {ratio:.2e}")
    assert ratio <= PROPERTY_REL
    a = (dq * q2d).sum(dim=(2, 3))
    b = (dk * k2d).sum(dim=(2, 3))
    scale = (dq * q2d).sum(dim=3).abs().sum(dim=2)
    rel = ((a - b).abs() / scale).max().item()
    _log(f"[fullsize] {name}: max_h |<dQ2,Q2> - <dK2,K2>| / sum_i |dQ2_i . Q2_i| = {rel:.2e}")
    assert rel <= PROPERTY_REL
    del dq, dk, q2d, k2d

    # --- sampled rows of three heads against the oracle
    rng = np.random.default_rng(w.seed)
    heads = sorted({(0, 0), (w.B - 1, w.H - 1), (int(rng.integers(w.B)), int(rng.integers(w.H)))})
    args = (d["Q1"], d["K1"], d["Q2"], d["K2"], w.s1, w.s2, causal, 0)
    for b_, h_ in heads:
        rows = _sample_rows(w.n_q, rng)
        rk, r1, r2 = oracle.forward_rows(*args, b_, h_, rows)
        ridx = torch.as_tensor(rows, device=kl.device)
        check_rows("kl", kl[b_, h_, ridx].cpu().numpy(), rk)
        check_rows("lse1", l1[b_, h_, ridx].cpu().numpy(), r1)
        check_rows("lse2", l2[b_, h_, ridx].cpu().numpy(), r2)
        _, rq2 = oracle.dq_rows(*args, b_, h_, rows, d["g"][b_, h_, rows])
        e = check_grad("dq2", dq2[b_, h_, ridx].cpu().numpy(), rq2)
        _log(f"[fullsize] {name}: head ({b_},{h_}) {rows.size} rows ok, dQ2 rel L2 {e:.2e}")

    # --- sampled keys of one head
    b_, h_ = heads[-1]
    keys = _sample_keys(w, causal, rng, full_stats_ok)
    t1 = time.time()
    _, rk2 = oracle.dk_rows(*args, b_, h_, keys, d["g"][b_, h_], row_block=512)
    kidx = torch.as_tensor(keys, device=kl.device)
    e = check_grad("dk2", dk2[b_, h_, kidx].cpu().numpy(), rk2)
    assert e <= GRAD_REL_L2
    _log(f"[fullsize] {name}: head ({b_},{h_}) {keys.size} keys ok, dK2 rel L2 {e:.2e} "
         f"(oracle {time.time() - t1:.1f} s); total {time.time() - t0:.1f} s")


def test_fullsize_distill_causal(gpu_lib):
    _run_full(gpu_lib, "distill", True, full_stats_ok=True)


def test_fullsize_mid_noncausal(gpu_lib):
    _run_full(gpu_lib, "mid", False, full_stats_ok=True)


def test_fullsize_mid_causal(gpu_lib):
    """The mid workload with the causal mask: 32 heads of 16384 rows make 2048
    workgroups of 256 rows, so this runs the eight-wave causal forward and the
    dQ/dK kernels at the shape the benchmark times."""
    _run_full(gpu_lib, "mid", True, full_stats_ok=True)


def test_fullsize_long_causal(gpu_lib):
    _run_full(gpu_lib, "long", True, full_stats_ok=False)


def test_fullsize_indexer_causal(gpu_lib):
    _run_full(gpu_lib, "indexer", True, full_stats_ok=False)


@pytest.mark.parametrize("n_q", [1, 16, 64])
def test_fullsize_decode_split_and_fused(gpu_lib, n_q):
    """The decode-like shapes that the split-K and backward-strategy figures
    time (16 heads, N_K = 65536, d1 = d2 = 128, non-causal), through the
    adaptive paths: the split-K forward and the fused backward the rule picks.
    Every query row of three heads and sampled keys of one head against the
    oracle; the fused gradients against the separate kernels' on all heads."""
    import torch
    t0 = time.time()
    d = inputs.make("mid", B=16, H=1, n_q=n_q, n_k=65536)
    w = d["w"]
    _log(f"[fullsize] decode n_q={n_q}: B={w.B} H={w.H} NK={w.n_k} d={w.d1}")
    q1, k1, q2, k2 = upload(d)
    g = to_gpu_f32(d["g"])
    assert gpu_lib.split_count(w.B, w.H, n_q, w.n_k, w.d1, w.d2) > 1
    assert gpu_lib.bwd_choose(w.B, w.H, n_q, w.n_k, w.d1, w.d2) == "fused"
    kl, l1, l2 = gpu_lib.fwd_split(q1, k1, q2, k2, w.s1, w.s2, False, 0, splits="auto")
    want = ("dq2", "dk2")
    fused = gpu_lib.bwd(q1, k1, q2, k2, kl, l1, l2, g, w.s1, w.s2, False, 0, want=want, strategy="auto")
    sep = gpu_lib.bwd(q1, k1, q2, k2, kl, l1, l2, g, w.s1, w.s2, False, 0, want=want, strategy="separate")
    torch.cuda.synchronize()
    _log(f"[fullsize] decode n_q={n_q}: GPU passes {time.time() - t0:.1f} s")
    assert float(kl.min()) >= -KL_ATOL
    for name, f, s in zip(("dq2", "dk2"), fused[2:], sep[2:]):
        rel = float((f.double() - s.double()).norm() / s.double().norm())
        assert rel <= 1e-5, (name, rel)

    rng = np.random.default_rng(w.seed + n_q)
    args = (d["Q1"], d["K1"], d["Q2"], d["K2"], w.s1, w.s2, False, 0)
    rows = np.arange(n_q)
    for b_ in sorted({0, w.B - 1, int(rng.integers(w.B))}):
        rk, r1, r2 = oracle.forward_rows(*args, b_, 0, rows)
        check_rows("kl", kl[b_, 0].cpu().numpy(), rk)
        check_rows("lse1", l1[b_, 0].cpu().numpy(), r1)
        check_rows("lse2", l2[b_, 0].cpu().numpy(), r2)
        _, rq2 = oracle.dq_rows(*args, b_, 0, rows, d["g"][b_, 0, rows])
        check_grad("dq2", fused[2][b_, 0].cpu().numpy(), rq2)
    b_ = w.B - 1
    keys = np.unique(np.concatenate([[0, 1, 127, 128, w.n_k // 2, w.n_k - 1], rng.choice(w.n_k, 40, replace=False)]))
    _, rk2 = oracle.dk_rows(*args, b_, 0, keys, d["g"][b_, 0])
    kidx = torch.as_tensor(keys, device=kl.device)
    e = check_grad("dk2", fused[3][b_, 0, kidx].cpu().numpy(), rk2)
    _log(f"[fullsize] decode n_q={n_q}: rows and {keys.size} keys ok, dK2 rel L2 {e:.2e}; "
         f"total {time.time() - t0:.1f} s")


def test_maximum_key_extent(gpu_lib):
    """The largest key count the boundary accepts at d1 = d2 = 256: one head's
    fp32 dK slab is just under 4 GiB (2^32 - 1024 bytes), the limit of the
    32-bit slab offsets. Few query rows, so the adaptive paths run (split-K
    forward, fused backward); both agree with the single-pass forward and the
    separate backward kernels, and every row and sampled keys (first, around
    2^21, the ragged last tile) match the oracle."""
    import torch
    t0 = time.time()
    n_k = 4194303
    assert gpu_lib.lib.streamkl_fwd(None, None, None, None, 1, 1, 8, n_k + 1, 256, 256, 0.0625, 0.0625, 0, 0,
                                    None, None, None, None) == gpu_lib.ERR_UNSUPPORTED
    d = inputs.make("tiny", B=1, H=1, n_q=8, n_k=n_k, d1=256, d2=256, s1=0.0625, s2=0.0625)
    w = d["w"]
    _log(f"[fullsize] max extent: NK={n_k} d=256, inputs {time.time() - t0:.1f} s")
    q1, k1, q2, k2 = upload(d)
    g = to_gpu_f32(d["g"])
    want = ("dq2", "dk2")
    for causal in (False, True):
        kl, l1, l2 = gpu_lib.fwd_split(q1, k1, q2, k2, w.s1, w.s2, causal, 0, splits="auto")
        one = gpu_lib.fwd(q1, k1, q2, k2, w.s1, w.s2, causal, 0)
        grads = gpu_lib.bwd(q1, k1, q2, k2, kl, l1, l2, g, w.s1, w.s2, causal, 0, want=want, strategy="auto")
        torch.cuda.synchronize()
        for a, b in zip((kl, l1, l2), one):
            assert torch.allclose(a, b, rtol=2e-5, atol=2e-5)
        sep = gpu_lib.bwd(q1, k1, q2, k2, kl, l1, l2, g, w.s1, w.s2, causal, 0, want=want, strategy="separate")
        torch.cuda.synchronize()
        # the same fp32 sums over 4M keys in two orders (atomics over key
        # blocks against one accumulator per row)
        for name, f, s in zip(want, grads[2:], sep[2:]):
            rel = float((f.double() - s.double()).norm() / s.double().norm())
            assert rel <= 1e-4, (name, rel)
        sep_dq2 = sep[2][0, 0].cpu().numpy()
        del sep
        _log(f"[fullsize] max extent causal={causal}: GPU passes done, {time.time() - t0:.1f} s")
        args = (d["Q1"], d["K1"], d["Q2"], d["K2"], w.s1, w.s2, causal, 0)
        rows = np.arange(w.n_q)
        rk, r1, r2 = oracle.forward_rows(*args, 0, 0, rows)
        check_rows("kl", kl[0, 0].cpu().numpy(), rk)
        check_rows("lse1", l1[0, 0].cpu().numpy(), r1)
        check_rows("lse2", l2[0, 0].cpu().numpy(), r2)
        check_rows("kl (single pass)", one[0][0, 0].cpu().numpy(), rk)
        _, rq2 = oracle.dq_rows(*args, 0, 0, rows, d["g"][0, 0, rows])
        check_grad("dq2", grads[2][0, 0].cpu().numpy(), rq2)
        check_grad("dq2 (separate)", sep_dq2, rq2)
        keys = np.array([0, 1, 2 ** 21 - 1, 2 ** 21, n_k - 33, n_k - 32, n_k - 2, n_k - 1])   # n_k - 1 = 2^22 - 1
        _, rk2 = oracle.dk_rows(*args, 0, 0, keys, d["g"][0, 0])
        e = check_grad("dk2", grads[3][0, 0, torch.as_tensor(keys, device=kl.device)].cpu().numpy(), rk2)
        _log(f"[fullsize] max extent causal={causal}: oracle ok, dK2 rel L2 {e:.2e}, {time.time() - t0:.1f} s")
        del grads


def test_maximum_query_extent(gpu_lib):
    """The largest query count the boundary accepts at d1 = d2 = 256 (one
    head's fp32 dQ slab just under 4 GiB), with 64 keys: the single-pass
    forward and the separate backward kernels (the rule's choice here) on
    sampled rows against the oracle, dK2 of every key, and the identity
    <dQ2, Q2> = <dK2, K2> over the whole head. Causal (bottom-right) leaves all
    but the last 64 rows without a visible key: KL 0, LSE -inf, zero dQ."""
    import torch
    t0 = time.time()
    n_q, n_k = 4194303, 64
    d = inputs.make("tiny", B=1, H=1, n_q=n_q, n_k=n_k, d1=256, d2=256, s1=0.0625, s2=0.0625)
    w = d["w"]
    _log(f"[fullsize] max query extent: NQ={n_q} NK={n_k} d=256, inputs {time.time() - t0:.1f} s")
    q1, k1, q2, k2 = upload(d)
    g = to_gpu_f32(d["g"])
    assert gpu_lib.bwd_choose(1, 1, n_q, n_k, 256, 256) == "separate"
    rng = np.random.default_rng(17)
    for causal in (False, True):
        kl, l1, l2 = gpu_lib.fwd(q1, k1, q2, k2, w.s1, w.s2, causal, 0)
        _, _, dq2, dk2 = gpu_lib.bwd(q1, k1, q2, k2, kl, l1, l2, g, w.s1, w.s2, causal, 0, want=("dq2", "dk2"))
        torch.cuda.synchronize()
        _log(f"[fullsize] max query extent causal={causal}: GPU passes done, {time.time() - t0:.1f} s")
        a = float((dq2.double() * q2.double()).sum())
        b = float((dk2.double() * k2.double()).sum())
        scale = float((dq2.double() * q2.double()).sum(dim=3).abs().sum())
        assert abs(a - b) <= PROPERTY_REL * scale, (a, b, scale)
        args = (d["Q1"], d["K1"], d["Q2"], d["K2"], w.s1, w.s2, causal, 0)
        rows = np.unique(np.concatenate([[0, 1, 2 ** 21, n_q - 65, n_q - 64, n_q - 2, n_q - 1],
                                         rng.choice(n_q, 24, replace=False)]))
        ridx = torch.as_tensor(rows, device=kl.device)
        rk, r1, r2 = oracle.forward_rows(*args, 0, 0, rows)
        check_rows("kl", kl[0, 0, ridx].cpu().numpy(), rk)
        check_rows("lse1", l1[0, 0, ridx].cpu().numpy(), r1)
        check_rows("lse2", l2[0, 0, ridx].cpu().numpy(), r2)
        _, rq2 = oracle.dq_rows(*args, 0, 0, rows, d["g"][0, 0, rows])
        check_grad("dq2", dq2[0, 0, ridx].cpu().numpy(), rq2)
        _, rk2 = oracle.dk_rows(*args, 0, 0, np.arange(n_k), d["g"][0, 0], row_block=1 << 20)
        e = check_grad("dk2", dk2[0, 0].cpu().numpy(), rk2)
        _log(f"[fullsize] max query extent causal={causal}: oracle ok, dK2 rel L2 {e:.2e}, {time.time() - t0:.1f} s")
        del kl, l1, l2, dq2, dk2


def test_fullsize_distill_reverse_all_gradients(gpu_lib):
    """The distillation workload (teacher d1 = 128, student d2 = 64, causal)
    in the reverse direction KL(P2 || P1) with all four gradients (the
    both-settings kernels), on sampled rows and keys of two heads."""
    import torch
    t0 = time.time()
    d = inputs.make("distill")
    w = d["w"]
    q1, k1, q2, k2 = upload(d)
    g = to_gpu_f32(d["g"])
    kl, l1, l2 = gpu_lib.fwd(q1, k1, q2, k2, w.s1, w.s2, True, 1)
    grads = gpu_lib.bwd(q1, k1, q2, k2, kl, l1, l2, g, w.s1, w.s2, True, 1, want=("dq1", "dk1", "dq2", "dk2"))
    torch.cuda.synchronize()
    _log(f"[fullsize] distill reverse: GPU passes {time.time() - t0:.1f} s")
    assert float(kl.min()) >= -KL_ATOL
    rng = np.random.default_rng(w.seed + 1)
    args = (d["Q1"], d["K1"], d["Q2"], d["K2"], w.s1, w.s2, True, 1)
    for b_, h_ in ((0, 0), (w.B - 1, w.H - 1)):
        rows = _sample_rows(w.n_q, rng, k=24)
        ridx = torch.as_tensor(rows, device=kl.device)
        rk, r1, r2 = oracle.forward_rows(*args, b_, h_, rows)
        check_rows("kl", kl[b_, h_, ridx].cpu().numpy(), rk)
        check_rows("lse1", l1[b_, h_, ridx].cpu().numpy(), r1)
        check_rows("lse2", l2[b_, h_, ridx].cpu().numpy(), r2)
        rq1, rq2 = oracle.dq_rows(*args, b_, h_, rows, d["g"][b_, h_, rows])
        check_grad("dq1", grads[0][b_, h_, ridx].cpu().numpy(), rq1)
        check_grad("dq2", grads[2][b_, h_, ridx].cpu().numpy(), rq2)
        keys = _sample_keys(w, True, rng, True, k=16)
        kidx = torch.as_tensor(keys, device=kl.device)
        rk1, rk2 = oracle.dk_rows(*args, b_, h_, keys, d["g"][b_, h_], row_block=512)
        check_grad("dk1", grads[1][b_, h_, kidx].cpu().numpy(), rk1)
        check_grad("dk2", grads[3][b_, h_, kidx].cpu().numpy(), rk2)
        _log(f"[fullsize] distill reverse: head ({b_},{h_}) ok, {time.time() - t0:.1f} s")
