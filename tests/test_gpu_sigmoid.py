"""GPU parity of the sigmoid-score path (streamkl_fwd_act / streamkl_bwd_act,
Sec. 3.1 "Generalizability beyond Softmax") against the fp64 oracle in
oracle/sigmoid_oracle.py, element by element on the seeded bf16 inputs:
the generalized KL and both row masses per row (row tolerance), every
gradient tensor (relative L2 and per-row bounds), over several tiles, ragged
and empty shapes, every head-dim pair, both directions, the workloads' value
distributions, and sampled rows of the full mid workload."""
import time

import numpy as np
import pytest

from oracle import sigmoid_oracle as so
from paper_2606_20005_amd import inputs
from parity_utils import check_grad, check_rows, to_gpu_f32, upload

pytestmark = pytest.mark.gpu

ALL = ("dq1", "dk1", "dq2", "dk2")


def run_case(sk, d, causal, direction, want=ALL, use_g=True):
    import torch
    w = d["w"]
    q1, k1, q2, k2 = upload(d)
    kl, m1, m2 = sk.fwd_act(q1, k1, q2, k2, w.s1, w.s2, causal, direction, "sigmoid")
    g_np = d["g"] if use_g else None
    g = to_gpu_f32(g_np) if use_g else None
    grads = sk.bwd(q1, k1, q2, k2, None, None, None, g, w.s1, w.s2, causal, direction, want=want,
                   activation="sigmoid")
    torch.cuda.synchronize()
    ref = so.backward(d["Q1"], d["K1"], d["Q2"], d["K2"], w.s1, w.s2, causal, direction, g_np)
    check_rows("kl", kl.cpu().numpy(), ref[0])
    check_rows("mass1", m1.cpu().numpy(), ref[1])
    check_rows("mass2", m2.cpu().numpy(), ref[2])
    for name, got, r in zip(ALL, grads, ref[3:]):
        if name in want:
            check_grad(name, got.cpu().numpy(), r)
        else:
            assert got is None


@pytest.mark.parametrize("direction", [0, 1])
@pytest.mark.parametrize("causal", [False, True])
def test_sigmoid_tiny_all_outputs(gpu_lib, causal, direction):
    run_case(gpu_lib, inputs.make("tiny"), causal, direction)


def test_sigmoid_identical_exact_zero(gpu_lib):
    import torch
    d = inputs.make("tiny", "identical")
    w = d["w"]
    q1, k1, q2, k2 = upload(d)
    for causal in (False, True):
        kl, _, _ = gpu_lib.fwd_act(q1, k1, q2, k2, w.s1, w.s2, causal, 0, "sigmoid")
        grads = gpu_lib.bwd(q1, k1, q2, k2, None, None, None, None, w.s1, w.s2, causal, 0, want=ALL,
                            activation="sigmoid")
        torch.cuda.synchronize()
        assert float(kl.abs().max()) == 0.0
        for t in grads:
            assert float(t.abs().max()) == 0.0


@pytest.mark.parametrize("nq,nk,causal", [
    (257, 257, False), (257, 257, True), (100, 300, True), (300, 100, True), (1, 1, False), (33, 129, True),
    (129, 33, False), (64, 1, True),
])
def test_sigmoid_ragged_shapes(gpu_lib, nq, nk, causal):
    run_case(gpu_lib, inputs.make("tiny", B=1, H=2, n_q=nq, n_k=nk), causal, 0)


@pytest.mark.parametrize("d1", [64, 128, 192, 256])
@pytest.mark.parametrize("d2", [64, 128, 192, 256])
def test_sigmoid_every_head_dim_pair(gpu_lib, d1, d2):
    d = inputs.make("tiny", B=1, H=1, n_q=160, n_k=200, d1=d1, d2=d2, s1=d1 ** -0.5, s2=d2 ** -0.5)
    run_case(gpu_lib, d, True, 0, want=("dq2", "dk2"))
    run_case(gpu_lib, d, False, 1, want=("dq1", "dk1"))


@pytest.mark.parametrize("want", [("dq2", "dk2"), ("dq1", "dk1"), ("dq2",), ("dk1",)])
def test_sigmoid_gradient_subsets_and_signed_g(gpu_lib, want):
    d = inputs.make("tiny", B=1, H=2, n_q=200, n_k=230, d1=128, d2=64, s1=128 ** -0.5)
    rng = np.random.default_rng(3)
    d["g"] = (d["g"] * rng.choice(np.float32([-1, 1]), size=d["g"].shape)).astype(np.float32)
    d["g"][..., ::17] = 0.0
    run_case(gpu_lib, d, True, 0, want=want)


def test_sigmoid_upstream_gradient_none_is_ones(gpu_lib):
    run_case(gpu_lib, inputs.make("tiny", n_q=130, n_k=190), True, 1, use_g=False)


@pytest.mark.parametrize("name,over,causal", [
    ("distill", dict(H=2, n_q=512, n_k=512), True),
    ("mid", dict(H=2, n_q=512, n_k=512), False),
    ("mid", dict(H=1024, n_q=256, n_k=256), True),
    ("long", dict(H=2, n_q=640, n_k=640), True),
    ("indexer", dict(H=2, n_q=128, n_k=2048), True),
])
def test_sigmoid_workload_structures_reduced(gpu_lib, name, over, causal):
    """Each workload's value distribution (the outlier logits of the long
    workload included) and masking; 1024 heads of 256 rows reach the
    eight-wave causal configuration."""
    d = inputs.make(name, **over)
    if d["w"].H > 8:      # check four heads of many against the oracle
        import torch
        w = d["w"]
        q1, k1, q2, k2 = upload(d)
        g = to_gpu_f32(d["g"])
        kl, m1, m2 = gpu_lib.fwd_act(q1, k1, q2, k2, w.s1, w.s2, causal, 0, "sigmoid")
        _, _, dq2, dk2 = gpu_lib.bwd(q1, k1, q2, k2, None, None, None, g, w.s1, w.s2, causal, 0,
                                     want=("dq2", "dk2"), activation="sigmoid")
        torch.cuda.synchronize()
        for h in (0, 1, 517, w.H - 1):
            sl = lambda x: x[:, h:h + 1]  # noqa: E731
            ref = so.backward(sl(d["Q1"]), sl(d["K1"]), sl(d["Q2"]), sl(d["K2"]), w.s1, w.s2, causal, 0, sl(d["g"]))
            check_rows("kl", kl[:, h:h + 1].cpu().numpy(), ref[0])
            check_rows("mass1", m1[:, h:h + 1].cpu().numpy(), ref[1])
            check_grad("dq2", dq2[:, h:h + 1].cpu().numpy(), ref[5])
            check_grad("dk2", dk2[:, h:h + 1].cpu().numpy(), ref[6])
        return
    run_case(gpu_lib, d, causal, 0)


def test_sigmoid_autograd(gpu_lib):
    import torch
    d = inputs.make("distill", H=2, n_q=256, n_k=256)
    w = d["w"]
    q1, k1, q2, k2 = upload(d)
    q2.requires_grad_(True)
    k2.requires_grad_(True)
    kl = gpu_lib.attention_kl(q1, k1, q2, k2, s1=w.s1, s2=w.s2, causal=True, activation="sigmoid")
    kl.mean().backward()
    torch.cuda.synchronize()
    n = kl.numel()
    ref = so.backward(d["Q1"], d["K1"], d["Q2"], d["K2"], w.s1, w.s2, True, 0, np.full(kl.shape, 1.0 / n))
    check_rows("kl", kl.detach().cpu().numpy(), ref[0])
    check_grad("dq2", q2.grad.float().cpu().numpy(), ref[5])
    check_grad("dk2", k2.grad.float().cpu().numpy(), ref[6])


def test_sigmoid_softmax_through_act_entry_point_is_fwd(gpu_lib):
    """activation = softmax through streamkl_fwd_act is streamkl_fwd, bit for bit."""
    import torch
    d = inputs.make("distill", H=2, n_q=300, n_k=300)
    w = d["w"]
    q1, k1, q2, k2 = upload(d)
    a = gpu_lib.fwd_act(q1, k1, q2, k2, w.s1, w.s2, True, 0, "softmax")
    b = gpu_lib.fwd(q1, k1, q2, k2, w.s1, w.s2, True, 0)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)


@pytest.mark.slow
def test_sigmoid_fullsize_mid_sampled(gpu_lib):
    """The mid workload at full size (32 heads, 16384 x 16384, d = 128,
    non-causal and causal): sampled rows of two heads (KL, masses, dQ2) and
    sampled keys of one head (dK2) against the oracle."""
    import torch
    t0 = time.time()
    d = inputs.make("mid")
    w = d["w"]
    q1, k1, q2, k2 = upload(d)
    g = to_gpu_f32(d["g"])
    rng = np.random.default_rng(w.seed + 5)
    for causal in (False, True):
        kl, m1, m2 = gpu_lib.fwd_act(q1, k1, q2, k2, w.s1, w.s2, causal, 0, "sigmoid")
        _, _, dq2, dk2 = gpu_lib.bwd(q1, k1, q2, k2, None, None, None, g, w.s1, w.s2, causal, 0,
                                     want=("dq2", "dk2"), activation="sigmoid")
        torch.cuda.synchronize()
        print(f"[sigmoid fullsize] causal={causal}: GPU passes {time.time() - t0:.1f} s", flush=True)
        assert bool(torch.isfinite(kl).all()) and float(kl.min()) >= -1e-3
        args = (d["Q1"], d["K1"], d["Q2"], d["K2"], w.s1, w.s2, causal, 0)
        for b_, h_ in ((0, 0), (0, w.H - 1)):
            rows = np.unique(np.concatenate([[0, 1, 255, 256, w.n_q - 1], rng.choice(w.n_q, 40, replace=False)]))
            ridx = torch.as_tensor(rows, device="cuda")
            rk, r1, r2 = so.forward_rows(*args, b_, h_, rows)
            check_rows("kl", kl[b_, h_, ridx].cpu().numpy(), rk)
            check_rows("mass1", m1[b_, h_, ridx].cpu().numpy(), r1)
            check_rows("mass2", m2[b_, h_, ridx].cpu().numpy(), r2)
            _, rq2 = so.dq_rows(*args, b_, h_, rows, d["g"][b_, h_, rows])
            check_grad("dq2", dq2[b_, h_, ridx].cpu().numpy(), rq2)
        keys = np.unique(np.concatenate([[0, 127, 128, w.n_k - 1], rng.choice(w.n_k, 20, replace=False)]))
        _, rk2 = so.dk_rows(*args, 0, 3, keys, d["g"][0, 3], row_block=1024)
        check_grad("dk2", dk2[0, 3, torch.as_tensor(keys, device="cuda")].cpu().numpy(), rk2)
        print(f"[sigmoid fullsize] causal={causal}: oracle ok, {time.time() - t0:.1f} s", flush=True)
