"""Helpers shared by the GPU parity tests: upload of the seeded bf16 inputs,
the oracle-side reference, and the tolerance checks.

Tolerances (fixed by the target of this implementation):
  per-row KL (and LSE):  |gpu - ref| <= 1e-3 + 1e-2 * |ref|
  each gradient tensor:  ||gpu - ref||_2 / ||ref||_2 <= 1e-2,
                         or max |gpu| <= 1e-6 when ref is identically 0.
Beside the tensor-level bound, every gradient row (a query row of dQ, a key
row of dK: the last axis is the head dim) must satisfy
  ||gpu_r - ref_r||_2 <= 5e-2 * ||ref_r||_2 + 1e-3 * rms_r ||ref_r||_2,
so that one wrong element, which moves the whole-tensor norm by well under
1e-2 in a large tensor, still fails its own row. The expected per-row error
is the bf16 rounding of dS before the second product, about 2^-9 of the row
norm; the small floor keeps rows whose reference is (nearly) zero from
failing on rounding alone.
"""
import numpy as np

KL_ATOL, KL_RTOL = 1e-3, 1e-2
GRAD_REL_L2 = 1e-2
GRAD_ZERO_ATOL = 1e-6
GRAD_ROW_REL_L2 = 5e-2
GRAD_ROW_FLOOR = 1e-3


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
    check_grad_rows(name, got, ref)
    return rel


def check_grad_rows(name, got, ref):
    """Per-row relative L2 bound (rows = all but the last axis)."""
    d = ref.shape[-1] if ref.ndim else 1
    g2 = got.reshape(-1, d)
    r2 = ref.reshape(-1, d)
    rn = np.linalg.norm(r2, axis=1)
    rms = float(np.sqrt(np.mean(rn ** 2))) if rn.size else 0.0
    err = np.linalg.norm(g2 - r2, axis=1)
    bound = GRAD_ROW_REL_L2 * rn + GRAD_ROW_FLOOR * rms
    bad = err > bound
    if np.any(bad):
        i = int(np.argmax(err - bound))
        raise AssertionError(f"{name}: {int(bad.sum())} rows over the per-row bound; worst flat row {i}: "
                             f"error {err[i]:.3e}, row norm {rn[i]:.3e}, bound {bound[i]:.3e}")
