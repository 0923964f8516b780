"""Helpers shared by the GPU parity tests: upload of the seeded bf16 inputs,
the oracle-side reference, and the tolerance checks.

Tolerances (fixed by the target of this implementation):
  per-row KL (and LSE):  |gpu - ref| <= 1e-3 + 1e-2 * |ref|
  each gradient tensor:  ||gpu - ref||_2 / ||ref||_2 <= 1e-2,
                         or max |gpu| <= 1e-6 when ref is identically 0.
"""
import numpy as np

KL_ATOL, KL_RTOL = 1e-3, 1e-2
GRAD_REL_L2 = 1e-2
GRAD_ZERO_ATOL = 1e-6


def to_gpu_bf16(x):
    import torch
    from paper_2606_20005_amd import inputs
    return torch.from_numpy(inputs.bf16_bits(x).view(np.int16)).view(torch.bfloat16).cuda()


def to_gpu_f32(x):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()


def upload(d):
    return tuple(to_gpu_bf16(d[k]) for k in ("Q1", "K1", "Q2", "K2"))


def check_rows(name, got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    both_ninf = np.isneginf(got) & np.isneginf(ref)
    assert np.array_equal(np.isneginf(got), np.isneginf(ref)), f"{name}: -inf pattern differs"
    g = np.where(both_ninf, 0.0, got)
    r = np.where(both_ninf, 0.0, ref)
    assert np.all(np.isfinite(g)), f"{name}: non-finite values"
    err = np.abs(g - r)
    bound = KL_ATOL + KL_RTOL * np.abs(r)
    worst = int(np.argmax(err - bound))
    assert np.all(err <= bound), f"{name}: max excess at flat index {worst}: got {g.flat[worst]} ref {r.flat[worst]}"
    return float(np.max(err)) if err.size else 0.0


def check_grad(name, got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{name}: non-finite values"
    nref = np.linalg.norm(ref)
    if nref == 0.0:
        m = float(np.max(np.abs(got))) if got.size else 0.0
        assert m <= GRAD_ZERO_ATOL, f"{name}: reference is 0, gpu max |g| = {m}"
        return m
    rel = float(np.linalg.norm(got - ref) / nref)
    assert rel <= GRAD_REL_L2, f"{name}: relative L2 error {rel:.3e}"
    return rel
