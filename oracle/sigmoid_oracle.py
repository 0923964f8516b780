"""Plain fp64 definition of the distillation divergence under sigmoid attention scores.

TEST INFRASTRUCTURE (see ``oracle/__init__.py``): imported only by tests,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py``.

The paper (Sec. 3.1, "Generalizability beyond Softmax") states that the
method extends to attention activations without softmax's global
normalisation (it names ReLU, sigmoid and tanh) and that these are simpler,
because no normaliser has to be maintained. It gives neither the scores nor
the divergence for that case. The reading implemented here:

* scores are the elementwise sigmoid of the scaled logits, with no
  normalisation over the keys:  A_t[j] = sigmoid(S_t[j]),  S_t = s_t q_t K_t^T;
* the row value is the generalized KL divergence (I-divergence) of the two
  non-negative score rows over the keys the row may attend,

      L = sum_j [ A1_j log(A1_j / A2_j) - A1_j + A2_j ],

  which is >= 0, is 0 exactly when A1 = A2, and equals eq:kl-def whenever
  both rows sum to 1 (the last two terms then cancel);
* direction REV swaps the roles: L = sum_j [A2 log(A2/A1) - A2 + A1];
* masked keys (causal, bottom-right alignment as for softmax) contribute
  nothing, so a row with no visible key has L = 0 and zero gradients;
* besides L, the row masses M_t = sum_j A_t[j] are reported (the
  normalisers softmax would have divided by);
* ReLU and tanh are not covered by this reading: tanh scores can be
  negative (no logarithm), and ReLU makes L infinite wherever A2 = 0 < A1.

Logit gradients of g_i L_i (d/dS sigmoid(S) = A (1 - A)), FWD:

    dS1 = g A1 (1 - A1) (log A1 - log A2),     dS2 = g (A2 - A1) (1 - A2),

and REV with the roles of 1 and 2 swapped. No saved row statistic is needed.
Then dq_t = s_t dS_t K_t and dK_t = s_t dS_t^T q_t as for softmax.

Everything here is the plain definition, row block by row block, with the
sigmoid and its logarithm formed in the numerically stable way
(log sigmoid(S) = -log(1 + e^{-S}) for S >= 0 and S - log(1 + e^{S}) below).
"""
from __future__ import annotations

import numpy as np

from .kl_oracle import FWD, REV, _f32, _head, allowed_mask


def _check_direction(direction):
    if direction not in (FWD, REV):
        raise ValueError("direction must be 0 (first slot: teacher) or 1 (first slot: student)")


def sigmoid(S):
    """1 / (1 + e^{-S}) without overflow."""
    S = np.asarray(S, dtype=np.float64)
    e = np.exp(-np.abs(S))
    return np.where(S >= 0, 1.0 / (1.0 + e), e / (1.0 + e))


def log_sigmoid(S):
    """log sigmoid(S) without overflow or cancellation."""
    S = np.asarray(S, dtype=np.float64)
    return np.minimum(S, 0.0) - np.log1p(np.exp(-np.abs(S)))


def generalized_kl(p, q):
    """sum_j [p_j log(p_j / q_j) - p_j + q_j] over the last axis, p, q > 0."""
    p = np.asarray(p, dtype=np.float64)
    q = np.asarray(q, dtype=np.float64)
    return (p * (np.log(p) - np.log(q)) - p + q).sum(axis=-1)


def _rows(q1, k1, q2, k2, s1, s2, rows, n_q, causal):
    """Masked scores of the given rows of one head: mask, A1, A2 (0 where masked), log A1, log A2."""
    n_k = k1.shape[0]
    mask = allowed_mask(rows, n_q, n_k, causal)
    S1 = s1 * (q1 @ k1.T)
    S2 = s2 * (q2 @ k2.T)
    return dict(mask=mask, A1=np.where(mask, sigmoid(S1), 0.0), A2=np.where(mask, sigmoid(S2), 0.0),
                lA1=np.where(mask, log_sigmoid(S1), 0.0), lA2=np.where(mask, log_sigmoid(S2), 0.0))


def _row_values(rd, direction):
    """L and the two masses of each row (the divergence summed over allowed keys only)."""
    if direction == FWD:
        Aa, Ab, la, lb = rd["A1"], rd["A2"], rd["lA1"], rd["lA2"]
    else:
        Aa, Ab, la, lb = rd["A2"], rd["A1"], rd["lA2"], rd["lA1"]
    term = np.where(rd["mask"], Aa * (la - lb) - Aa + Ab, 0.0)
    return term.sum(axis=1), rd["A1"].sum(axis=1), rd["A2"].sum(axis=1)


def _logit_grads(rd, g, direction):
    """dS1, dS2 of g_i L_i (see the module docstring); 0 where masked."""
    A1, A2, mask = rd["A1"], rd["A2"], rd["mask"]
    g = np.asarray(g, dtype=np.float64)[:, None]
    if direction == FWD:
        dS1 = g * A1 * (1.0 - A1) * (rd["lA1"] - rd["lA2"])
        dS2 = g * (A2 - A1) * (1.0 - A2)
    else:
        dS2 = g * A2 * (1.0 - A2) * (rd["lA2"] - rd["lA1"])
        dS1 = g * (A1 - A2) * (1.0 - A1)
    return np.where(mask, dS1, 0.0), np.where(mask, dS2, 0.0)


def forward_rows(Q1, K1, Q2, K2, s1, s2, causal, direction, b, h, rows):
    """L, M1, M2 of the query rows ``rows`` of head (b, h) (each row needs only its own scores)."""
    _check_direction(direction)
    s1, s2 = _f32(s1), _f32(s2)
    rows = np.asarray(rows, dtype=np.int64).reshape(-1)
    n_q = Q1.shape[2]
    rd = _rows(_head(Q1, b, h)[rows], _head(K1, b, h), _head(Q2, b, h)[rows], _head(K2, b, h), s1, s2, rows, n_q,
               causal)
    return _row_values(rd, direction)


def dq_rows(Q1, K1, Q2, K2, s1, s2, causal, direction, b, h, rows, g):
    """dQ1[rows], dQ2[rows] of head (b, h); g holds one value per row."""
    _check_direction(direction)
    s1, s2 = _f32(s1), _f32(s2)
    rows = np.asarray(rows, dtype=np.int64).reshape(-1)
    n_q = Q1.shape[2]
    k1h, k2h = _head(K1, b, h), _head(K2, b, h)
    rd = _rows(_head(Q1, b, h)[rows], k1h, _head(Q2, b, h)[rows], k2h, s1, s2, rows, n_q, causal)
    dS1, dS2 = _logit_grads(rd, g, direction)
    return s1 * (dS1 @ k1h), s2 * (dS2 @ k2h)


def dk_rows(Q1, K1, Q2, K2, s1, s2, causal, direction, b, h, keys, g, row_block=256):
    """dK1[keys], dK2[keys] of head (b, h), summed over every row (g: [N_Q])."""
    _check_direction(direction)
    s1, s2 = _f32(s1), _f32(s2)
    keys = np.asarray(keys, dtype=np.int64).reshape(-1)
    n_q, n_k = Q1.shape[2], K1.shape[2]
    q1h, q2h = _head(Q1, b, h), _head(Q2, b, h)
    k1c, k2c = _head(K1, b, h)[keys], _head(K2, b, h)[keys]
    g = np.asarray(g, dtype=np.float64).reshape(-1)
    dk1 = np.zeros((keys.size, q1h.shape[1]))
    dk2 = np.zeros((keys.size, q2h.shape[1]))
    for r0 in range(0, n_q, row_block):
        rows = np.arange(r0, min(n_q, r0 + row_block))
        mask = allowed_mask(rows, n_q, n_k, causal)[:, keys]
        S1 = s1 * (q1h[rows] @ k1c.T)
        S2 = s2 * (q2h[rows] @ k2c.T)
        rd = dict(mask=mask, A1=np.where(mask, sigmoid(S1), 0.0), A2=np.where(mask, sigmoid(S2), 0.0),
                  lA1=np.where(mask, log_sigmoid(S1), 0.0), lA2=np.where(mask, log_sigmoid(S2), 0.0))
        dS1, dS2 = _logit_grads(rd, g[rows], direction)
        dk1 += s1 * (dS1.T @ q1h[rows])
        dk2 += s2 * (dS2.T @ q2h[rows])
    return dk1, dk2


def forward(Q1, K1, Q2, K2, s1, s2, causal=False, direction=FWD, row_block=256):
    """L, M1, M2 as [B, H, N_Q] fp64 arrays for every row of every head."""
    B, H, n_q = Q1.shape[:3]
    out = [np.empty((B, H, n_q)) for _ in range(3)]
    for b in range(B):
        for h in range(H):
            for r0 in range(0, n_q, row_block):
                rows = np.arange(r0, min(n_q, r0 + row_block))
                vals = forward_rows(Q1, K1, Q2, K2, s1, s2, causal, direction, b, h, rows)
                for o, v in zip(out, vals):
                    o[b, h, rows] = v
    return tuple(out)


def backward(Q1, K1, Q2, K2, s1, s2, causal=False, direction=FWD, dkl=None, row_block=256):
    """(L, M1, M2, dQ1, dK1, dQ2, dK2) for every head, fp64; dkl: [B, H, N_Q] upstream gradient (None: ones)."""
    _check_direction(direction)
    s1, s2 = _f32(s1), _f32(s2)
    B, H, n_q = Q1.shape[:3]
    if dkl is None:
        dkl = np.ones((B, H, n_q))
    L, M1, M2 = (np.empty((B, H, n_q)) for _ in range(3))
    dQ1, dQ2 = np.zeros(Q1.shape), np.zeros(Q2.shape)
    dK1, dK2 = np.zeros(K1.shape), np.zeros(K2.shape)
    for b in range(B):
        for h in range(H):
            q1h, k1h, q2h, k2h = _head(Q1, b, h), _head(K1, b, h), _head(Q2, b, h), _head(K2, b, h)
            for r0 in range(0, n_q, row_block):
                rows = np.arange(r0, min(n_q, r0 + row_block))
                rd = _rows(q1h[rows], k1h, q2h[rows], k2h, s1, s2, rows, n_q, causal)
                L[b, h, rows], M1[b, h, rows], M2[b, h, rows] = _row_values(rd, direction)
                dS1, dS2 = _logit_grads(rd, np.asarray(dkl[b, h, rows], dtype=np.float64), direction)
                dQ1[b, h, rows] = s1 * (dS1 @ k1h)
                dQ2[b, h, rows] = s2 * (dS2 @ k2h)
                dK1[b, h] += s1 * (dS1.T @ q1h[rows])
                dK2[b, h] += s2 * (dS2.T @ q2h[rows])
    return L, M1, M2, dQ1, dK1, dQ2, dK2
