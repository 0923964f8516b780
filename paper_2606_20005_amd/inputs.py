"""Seeded synthetic inputs for the attention-distillation KL workloads.

This module holds none of the method's arithmetic: it only draws Gaussian
tensors from fixed seeds, rounds them to bf16 (round to nearest even) and
applies the structure each workload asks for. Both the GPU path and the fp64
oracle are fed the very same bf16-valued arrays (the oracle lifts them exactly
to fp64), so a mismatch can only come from the arithmetic.

The paper evaluates on synthetic shapes only (bsz 16/32, contexts 4K-512K,
d = 128, causal and non-causal; Sec. 6.1) and names no dataset; the workloads
below follow those shapes:

    tiny     B=1 H=1  N_Q=N_K=256     d1=d2=64     s=1/8              non-causal
    distill  B=2 H=16 N_Q=N_K=4096    d1=128 d2=64 s1=1/sqrt(128) s2=1/8  causal
    mid      B=1 H=32 N_Q=N_K=16384   d1=d2=128    s=1/sqrt(128)      non-causal (causal also run)
             Q2 = bf16(Q1 + 0.3*eps) and K2 = K1 (correlated distributions)
    long     B=1 H=32 N_Q=N_K=65536   d1=128 d2=64 s1=1/sqrt(128) s2=1/8  causal
             channels {5, 21, 37, 53} of all four tensors scaled by 8 (outlier logits)
    indexer  B=1 H=8  N_Q=8192 N_K=131072 d1=192 d2=64 s1=1/sqrt(192) s2=1/8
             causal by absolute position (the queries are the last 8192 tokens)

Seeds: seed = 2606200050 + workload id; one child stream per tensor from
``np.random.SeedSequence(seed).spawn(6)`` in the order Q1, K1, Q2, K2, eps, g.
The upstream gradient g is U[0.5, 1.5) per row.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, replace

import numpy as np

SEED_BASE = 2606_20005 * 10
OUTLIER_CHANNELS = (5, 21, 37, 53)
OUTLIER_SCALE = 8.0


@dataclass(frozen=True)
class Workload:
    name: str
    wid: int
    B: int
    H: int
    n_q: int
    n_k: int
    d1: int
    d2: int
    s1: float
    s2: float
    causal: bool
    structure: str = "independent"   # independent | correlated | outliers

    @property
    def seed(self) -> int:
        return SEED_BASE + self.wid


WORKLOADS = {
    "tiny": Workload("tiny", 1, 1, 1, 256, 256, 64, 64, 1 / 8, 1 / 8, False),
    "distill": Workload("distill", 2, 2, 16, 4096, 4096, 128, 64, 1 / math.sqrt(128), 1 / 8, True),
    "mid": Workload("mid", 3, 1, 32, 16384, 16384, 128, 128, 1 / math.sqrt(128), 1 / math.sqrt(128),
                    False, "correlated"),
    "long": Workload("long", 4, 1, 32, 65536, 65536, 128, 64, 1 / math.sqrt(128), 1 / 8, True, "outliers"),
    "indexer": Workload("indexer", 5, 1, 8, 8192, 131072, 192, 64, 1 / math.sqrt(192), 1 / 8, True),
}


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); returns float32.

    Inputs are finite Gaussian draws, so NaN handling is not needed.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)
    return r.view(np.float32)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """The uint16 bit patterns of bf16-valued float32 data (exact, no rounding)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    if np.any(u & np.uint32(0xFFFF)):
        raise ValueError("array holds values that are not bf16-representable")
    return (u >> np.uint32(16)).astype(np.uint16)


def _normal(ss, shape):
    return np.random.default_rng(ss).standard_normal(shape, dtype=np.float32)


def make(w: Workload | str, variant: str = "base", **overrides) -> dict:
    """Generate the inputs of a workload.

    variant: "base"; "identical" (Q2 = Q1, K2 = K1, s2 = s1: KL = 0);
    "q1zero" (Q1 = 0: P1 uniform over the allowed keys).
    overrides: any Workload field (e.g. n_q=257, causal=True) for edge shapes.
    Returns a dict with the Workload ``w`` and float32 bf16-valued arrays
    Q1, K1 [B,H,N_Q|N_K,d1], Q2, K2 [..,d2] and g [B,H,N_Q].
    """
    if isinstance(w, str):
        w = WORKLOADS[w]
    if overrides:
        w = replace(w, **overrides)
    if w.structure == "correlated" and w.d1 != w.d2:
        raise ValueError("correlated structure needs d1 == d2")
    ss = np.random.SeedSequence(w.seed).spawn(6)
    q_shape1 = (w.B, w.H, w.n_q, w.d1)
    k_shape1 = (w.B, w.H, w.n_k, w.d1)
    q_shape2 = (w.B, w.H, w.n_q, w.d2)
    k_shape2 = (w.B, w.H, w.n_k, w.d2)
    Q1 = round_bf16(_normal(ss[0], q_shape1))
    K1 = round_bf16(_normal(ss[1], k_shape1))
    if w.structure == "correlated":
        Q2 = round_bf16(Q1 + np.float32(0.3) * _normal(ss[4], q_shape2))
        K2 = K1.copy()
    else:
        Q2 = round_bf16(_normal(ss[2], q_shape2))
        K2 = round_bf16(_normal(ss[3], k_shape2))
    if w.structure == "outliers":
        for X in (Q1, K1, Q2, K2):
            ch = [c for c in OUTLIER_CHANNELS if c < X.shape[-1]]
            X[..., ch] *= np.float32(OUTLIER_SCALE)   # exact: a power of two
    g = np.random.default_rng(ss[5]).uniform(0.5, 1.5, size=(w.B, w.H, w.n_q)).astype(np.float32)
    if variant == "identical":
        if w.d1 != w.d2:
            raise ValueError("identical variant needs d1 == d2")
        Q2, K2 = Q1.copy(), K1.copy()
        w = replace(w, s2=w.s1)
    elif variant == "q1zero":
        Q1 = np.zeros_like(Q1)
    elif variant != "base":
        raise ValueError(f"unknown variant {variant!r}")
    return dict(w=w, Q1=Q1, K1=K1, Q2=Q2, K2=K2, g=g)
