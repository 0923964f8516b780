"""GPU parity of the fused backward (Sec. 4.2, one key-owned kernel, dQ by fp32
atomics) against the fp64 oracle, its agreement with the separate kernels,
and the adaptive strategy selection."""
import numpy as np
import pytest

import oracle
from paper_2606_20005_amd import inputs
from parity_utils import check_grad, check_rows, to_gpu_f32, upload

pytestmark = pytest.mark.gpu

ALL = ("dq1", "dk1", "dq2", "dk2")


def run_fused(sk, d, causal, direction, want, strategy="fused", out=None):
    import torch
    w = d["w"]
    q1, k1, q2, k2 = upload(d)
    kl, l1, l2 = sk.fwd(q1, k1, q2, k2, w.s1, w.s2, causal, direction)
    g = to_gpu_f32(d["g"])
    grads = sk.bwd(q1, k1, q2, k2, kl, l1, l2, g, w.s1, w.s2, causal, direction, want=want, out=out,
                   strategy=strategy)
    torch.cuda.synchronize()
    return grads, (q1, k1, q2, k2, kl, l1, l2, g)


def check_against_oracle(d, causal, direction, want, grads):
    w = d["w"]
    ref = oracle.backward(d["Q1"], d["K1"], d["Q2"], d["K2"], w.s1, w.s2, causal, direction, d["g"])
    for name, got, r in zip(ALL, grads, ref[3:]):
        if name in want:
            check_grad(name, got.cpu().numpy(), r)
        else:
            assert got is None


@pytest.mark.parametrize("nq,nk,causal", [
    (1, 4000, False),      # one row, ragged key tail, 32 key blocks add into it
    (16, 4096, False),     # decode-like
    (16, 4096, True),      # bottom-right causal: the last key blocks see only the last rows
    (100, 1000, True),     # several query tiles, ragged on both sides
    (257, 257, False),     # N_Q = N_K, ragged
    (257, 257, True),
    (300, 100, True),      # rows with no visible key (N_Q > N_K)
    (64, 1, False),        # one key
])
def test_fused_matches_oracle(gpu_lib, nq, nk, causal):
    d = inputs.make("tiny", B=2, H=2, n_q=nq, n_k=nk)
    grads, _ = run_fused(gpu_lib, d, causal, 0, ("dq2", "dk2"))
    check_against_oracle(d, causal, 0, ("dq2", "dk2"), grads)


@pytest.mark.parametrize("d1,d2", [(64, 64), (128, 128), (128, 64), (192, 64), (64, 256), (256, 128)])
def test_fused_head_dims(gpu_lib, d1, d2):
    d = inputs.make("tiny", B=1, H=2, n_q=96, n_k=700, d1=d1, d2=d2, s1=d1 ** -0.5, s2=d2 ** -0.5)
    for causal, direction in ((True, 0), (False, 1)):
        grads, _ = run_fused(gpu_lib, d, causal, direction, ("dq2", "dk2"))
        check_against_oracle(d, causal, direction, ("dq2", "dk2"), grads)


@pytest.mark.parametrize("want", [("dq1", "dk1"), ALL, ("dq2",), ("dq1", "dk2"), ("dq2", "dk1")])
@pytest.mark.parametrize("direction", [0, 1])
def test_fused_gradient_subsets(gpu_lib, want, direction):
    d = inputs.make("tiny", B=1, H=1, n_q=70, n_k=600, d1=128, d2=64, s1=128 ** -0.5)
    grads, _ = run_fused(gpu_lib, d, True, direction, want)
    check_against_oracle(d, True, direction, want, grads)


def test_fused_agrees_with_separate(gpu_lib):
    """Same logit gradients, same bf16 rounding of dS: dK and dQ agree up to the
    order of the fp32 sums (the fused kernel visits each key block's query
    tiles in a rotated order and adds dQ with atomics)."""
    import torch
    d = inputs.make("distill", H=2, n_q=1000, n_k=2048)   # 32 query tiles per key block
    grads_f, (q1, k1, q2, k2, kl, l1, l2, g) = run_fused(gpu_lib, d, True, 0, ALL)
    w = d["w"]
    grads_s = gpu_lib.bwd(q1, k1, q2, k2, kl, l1, l2, g, w.s1, w.s2, True, 0, want=ALL, strategy="separate")
    torch.cuda.synchronize()
    for name, f, s in zip(ALL, grads_f, grads_s):
        rel = float((f.double() - s.double()).norm() / s.double().norm())
        assert rel <= 1e-5, (name, rel)


def test_fused_zeroes_dq_first(gpu_lib):
    """dQ accumulates by atomics: preallocated outputs holding NaN are overwritten."""
    import torch
    d = inputs.make("tiny", B=1, H=2, n_q=40, n_k=900)
    w = d["w"]
    out = {"dq2": torch.full((1, 2, 40, w.d2), float("nan"), device="cuda"),
           "dk2": torch.full((1, 2, 900, w.d2), float("nan"), device="cuda")}
    grads, _ = run_fused(gpu_lib, d, False, 0, ("dq2", "dk2"), out=out)
    assert grads[2].data_ptr() == out["dq2"].data_ptr()
    check_against_oracle(d, False, 0, ("dq2", "dk2"), grads)


def test_fused_repeatable_up_to_sum_order(gpu_lib):
    import torch
    d = inputs.make("tiny", B=2, H=2, n_q=16, n_k=8192)
    a, args = run_fused(gpu_lib, d, False, 0, ("dq2", "dk2"))
    b, _ = run_fused(gpu_lib, d, False, 0, ("dq2", "dk2"))
    assert torch.equal(a[3], b[3])
    assert torch.allclose(a[2], b[2], rtol=1e-5, atol=1e-7)


def test_auto_strategy_follows_the_rule(gpu_lib):
    """'auto' gives the result of the strategy bwd_choose names."""
    import torch
    assert gpu_lib.bwd_choose(2, 2, 16, 4096, 64, 64) == "fused"
    assert gpu_lib.bwd_choose(2, 2, 512, 1024, 64, 64) == "separate"
    for nq, nk in ((16, 4096), (512, 1024)):
        d = inputs.make("tiny", B=2, H=2, n_q=nq, n_k=nk)
        auto, _ = run_fused(gpu_lib, d, True, 0, ("dq2", "dk2"), strategy="auto")
        pick, _ = run_fused(gpu_lib, d, True, 0, ("dq2", "dk2"),
                            strategy=gpu_lib.bwd_choose(2, 2, nq, nk, 64, 64))
        assert torch.equal(auto[3], pick[3])
        assert torch.allclose(auto[2], pick[2], rtol=1e-5, atol=1e-7)


def test_autograd_auto_strategy(gpu_lib):
    import torch
    d = inputs.make("tiny", B=2, H=2, n_q=8, n_k=2048)
    w = d["w"]
    q1, k1, q2, k2 = (t.clone().requires_grad_(True) for t in upload(d))
    assert gpu_lib.bwd_choose(2, 2, 8, 2048, 64, 64) == "fused"
    kl = gpu_lib.attention_kl(q1, k1, q2, k2, s1=w.s1, s2=w.s2, bwd_strategy="auto")
    kl.sum().backward()
    torch.cuda.synchronize()
    ref = oracle.backward(d["Q1"], d["K1"], d["Q2"], d["K2"], w.s1, w.s2, False, 0)
    check_rows("kl", kl.detach().cpu().numpy(), ref[0])
    for name, got, r in (("dq2", q2.grad, ref[5]), ("dk2", k2.grad, ref[6])):
        check_grad(name, got.float().cpu().numpy(), r)


def test_fused_unsupported_pairs_raise(gpu_lib):
    """All four gradients at d1 + d2 > 320 do not fit the fused kernel's LDS."""
    import torch
    d = inputs.make("tiny", B=1, H=1, n_q=32, n_k=256, d1=256, d2=256, s1=1 / 16, s2=1 / 16)
    with pytest.raises(gpu_lib.StreamKLError):
        run_fused(gpu_lib, d, False, 0, ALL)
    grads, _ = run_fused(gpu_lib, d, False, 0, ALL, strategy="auto")   # falls back to separate kernels
    check_against_oracle(d, False, 0, ALL, grads)
    torch.cuda.synchronize()
