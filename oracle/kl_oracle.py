"""Plain fp64 definition of the attention-distillation KL and its gradients.

TEST INFRASTRUCTURE (see ``oracle/__init__.py``): imported only by tests,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py``.

What is computed (paper Sec. 2.1, "KL Divergence"): for one query row with
logits S_t = s_t * q_t K_t^T (t = 1 teacher, t = 2 student) and attention
distributions P_t = softmax(S_t), the row value is

    L = KL(P1 || P2) = sum_j P1^j (log P1^j - log P2^j)          (eq:kl-def)

and the logit gradients are

    Setting 1 (P1 fixed):  dS2 = P2 - P1                          (eq:kl-case1)
    Setting 2 (P2 fixed):  dS1 = P1 * (r - L),  r = log P1 - log P2 (eq:kl-case2)

from which dq_t = s_t dS_t K_t and dK_t = s_t dS_t^T q_t (the factor s_t is
the chain rule through S_t = s_t q_t K_t^T). Both partials are exact at the
same time, so both are returned when asked for.

Everything here is the plain definition: P1 and P2 are materialised row block
by row block in fp64 from the bf16-valued inputs lifted exactly to fp64; the
KL is the direct sum of eq:kl-def (never the acc/l1 identity of
eq:kl-final, which is what the GPU path evaluates). A library matmul forms
the logits; nothing is fused, blocked across keys or reordered.

Readings where the paper is silent (the same list is kept with the design
notes of the repository):

* scale: S_t = s_t Q_t K_t^T with independent s1, s2 (the paper leaves
  the sqrt(d) factor out of its formulas); s_t is an fp32 argument of the operation, so it is
  rounded to fp32 before use.
* causal masking: bottom-right alignment. Query row i sits at absolute
  position N_K - N_Q + i and may attend keys j <= that position (inclusive);
  for N_Q = N_K this is j <= i.
* empty rows (only causal with N_Q > N_K): KL = 0, LSE = -inf, gradients 0.
* direction ``REV``: L = KL(P2 || P1), i.e. eq:kl-def with the roles of the
  two distributions swapped. LSE1 / LSE2 keep belonging to (Q1, K1) and
  (Q2, K2). The gradient of the distribution in the first KL slot then takes
  the Setting-2 form and the other the Setting-1 form.
* upstream gradient: one scalar g_i per row (Alg. 2 takes dL in R^{N_Q});
  every logit gradient is multiplied by g_i.
"""
from __future__ import annotations

import numpy as np

FWD = 0
REV = 1


def _f32(s: float) -> float:
    """The scale is an fp32 argument of the operation: round it to fp32."""
    return float(np.float32(s))


def allowed_mask(rows, n_q: int, n_k: int, causal: bool) -> np.ndarray:
    """Boolean [len(rows), n_k]; True where query row rows[r] may attend key j.

    Bottom-right causal alignment (reading, see module docstring).
    """
    rows = np.asarray(rows, dtype=np.int64).reshape(-1)
    if not causal:
        return np.ones((rows.size, n_k), dtype=bool)
    pos = rows + (n_k - n_q)
    return np.arange(n_k, dtype=np.int64)[None, :] <= pos[:, None]


def _logsumexp_rows(S: np.ndarray) -> np.ndarray:
    """Row-wise log(sum_j exp(S_j)) with -inf entries contributing 0.

    Rows whose entries are all -inf give -inf (empty rows).
    """
    m = S.max(axis=1)
    out = np.full(S.shape[0], -np.inf)
    ok = np.isfinite(m)
    if ok.any():
        Sm = S[ok] - m[ok, None]
        out[ok] = m[ok] + np.log(np.exp(Sm).sum(axis=1))
    return out


def _rows_quantities(q1, k1, q2, k2, s1, s2, rows, n_q, causal):
    """Masked logits, LSE and log-probabilities of the given rows of one head.

    q1: [len(rows), d1], k1: [N_K, d1], q2: [len(rows), d2], k2: [N_K, d2].
    Returns a dict with mask, S1, S2 (unmasked logits), lse1, lse2,
    logP1, logP2 (-inf where masked) and P1, P2 (0 where masked).
    """
    n_k = k1.shape[0]
    mask = allowed_mask(rows, n_q, n_k, causal)
    S1 = s1 * (q1 @ k1.T)
    S2 = s2 * (q2 @ k2.T)
    S1m = np.where(mask, S1, -np.inf)
    S2m = np.where(mask, S2, -np.inf)
    lse1 = _logsumexp_rows(S1m)
    lse2 = _logsumexp_rows(S2m)
    with np.errstate(invalid="ignore"):
        logP1 = np.where(mask, S1 - lse1[:, None], -np.inf)
        logP2 = np.where(mask, S2 - lse2[:, None], -np.inf)
    P1 = np.exp(logP1)
    P2 = np.exp(logP2)
    return dict(mask=mask, S1=S1, S2=S2, lse1=lse1, lse2=lse2,
                logP1=logP1, logP2=logP2, P1=P1, P2=P2)


def _row_kl(qd, direction):
    """Direct sum of eq:kl-def over the allowed keys of each row."""
    mask = qd["mask"]
    if direction == FWD:
        Pa, la, lb = qd["P1"], qd["logP1"], qd["logP2"]
    else:
        Pa, la, lb = qd["P2"], qd["logP2"], qd["logP1"]
    with np.errstate(invalid="ignore"):
        term = np.where(mask, Pa * (la - lb), 0.0)
    return term.sum(axis=1)


def _logit_grads(qd, kl, g, direction):
    """dS1, dS2 of g_i * L_i for each row (eq:kl-case1 / eq:kl-case2).

    FWD (L = KL(P1||P2)): dS2 = g (P2 - P1),  dS1 = g P1 (log P1 - log P2 - L).
    REV (L = KL(P2||P1)): dS1 = g (P1 - P2),  dS2 = g P2 (log P2 - log P1 - L).
    Masked entries are exactly 0.
    """
    mask = qd["mask"]
    P1, P2 = qd["P1"], qd["P2"]
    g = np.asarray(g, dtype=np.float64)[:, None]
    with np.errstate(invalid="ignore"):
        if direction == FWD:
            r = np.where(mask, qd["logP1"] - qd["logP2"], 0.0)
            dS2 = g * (P2 - P1)
            dS1 = g * P1 * np.where(mask, r - kl[:, None], 0.0)
        else:
            r = np.where(mask, qd["logP2"] - qd["logP1"], 0.0)
            dS1 = g * (P1 - P2)
            dS2 = g * P2 * np.where(mask, r - kl[:, None], 0.0)
    return dS1, dS2


def _head(X, b, h):
    return np.asarray(X[b, h], dtype=np.float64)


def _check_direction(direction):
    if direction not in (FWD, REV):
        raise ValueError("direction must be 0 (KL(P1||P2)) or 1 (KL(P2||P1))")


def forward_rows(Q1, K1, Q2, K2, s1, s2, causal, direction, b, h, rows):
    """KL, LSE1, LSE2 of the query rows ``rows`` of head (b, h).

    Q*: [B, H, N_Q, d*], K*: [B, H, N_K, d*] arrays (any float dtype; lifted
    to fp64). Each row needs only its own logits, so any subset is exact.
    """
    _check_direction(direction)
    s1, s2 = _f32(s1), _f32(s2)
    rows = np.asarray(rows, dtype=np.int64).reshape(-1)
    n_q = Q1.shape[2]
    q1 = _head(Q1, b, h)[rows]
    q2 = _head(Q2, b, h)[rows]
    qd = _rows_quantities(q1, _head(K1, b, h), q2, _head(K2, b, h), s1, s2, rows, n_q, causal)
    return _row_kl(qd, direction), qd["lse1"], qd["lse2"]


def logit_grads_rows(Q1, K1, Q2, K2, s1, s2, causal, direction, b, h, rows, g):
    """(dS1, dS2, kl) for the rows ``rows`` of head (b, h); g has one value per row."""
    _check_direction(direction)
    s1, s2 = _f32(s1), _f32(s2)
    rows = np.asarray(rows, dtype=np.int64).reshape(-1)
    n_q = Q1.shape[2]
    qd = _rows_quantities(_head(Q1, b, h)[rows], _head(K1, b, h),
                          _head(Q2, b, h)[rows], _head(K2, b, h), s1, s2, rows, n_q, causal)
    kl = _row_kl(qd, direction)
    dS1, dS2 = _logit_grads(qd, kl, g, direction)
    return dS1, dS2, kl


def dq_rows(Q1, K1, Q2, K2, s1, s2, causal, direction, b, h, rows, g):
    """dQ1[rows], dQ2[rows] of head (b, h): dq_t = s_t dS_t K_t (row-local)."""
    dS1, dS2, _ = logit_grads_rows(Q1, K1, Q2, K2, s1, s2, causal, direction, b, h, rows, g)
    return _f32(s1) * (dS1 @ _head(K1, b, h)), _f32(s2) * (dS2 @ _head(K2, b, h))


def head_stats_all_rows(Q1, K1, Q2, K2, s1, s2, causal, direction, b, h, row_block=256):
    """KL, LSE1, LSE2 for every query row of head (b, h), row block by row block."""
    n_q = Q1.shape[2]
    kl = np.empty(n_q)
    lse1 = np.empty(n_q)
    lse2 = np.empty(n_q)
    for r0 in range(0, n_q, row_block):
        rows = np.arange(r0, min(n_q, r0 + row_block))
        kl[rows], lse1[rows], lse2[rows] = forward_rows(
            Q1, K1, Q2, K2, s1, s2, causal, direction, b, h, rows)
    return kl, lse1, lse2


def dk_rows(Q1, K1, Q2, K2, s1, s2, causal, direction, b, h, keys, g, row_block=256):
    """dK1[keys], dK2[keys] of head (b, h): dK_t = s_t dS_t^T q_t summed over all rows.

    g: [N_Q] upstream gradient of this head. The LSE and KL of every row that
    can attend at least one of ``keys`` are computed first (a forward of those
    rows); then only the columns ``keys`` of dS are formed, row block by row
    block. Under the causal mask a row i sees key j only when
    j <= N_K - N_Q + i, so rows before min(keys) - (N_K - N_Q) have every
    sampled column masked: their terms are exactly zero and are not formed.
    """
    _check_direction(direction)
    s1, s2 = _f32(s1), _f32(s2)
    keys = np.asarray(keys, dtype=np.int64).reshape(-1)
    n_q, n_k = Q1.shape[2], K1.shape[2]
    r_first = max(0, int(keys.min()) - (n_k - n_q)) if causal else 0
    kl = np.zeros(n_q)
    lse1 = np.full(n_q, -np.inf)
    lse2 = np.full(n_q, -np.inf)
    for r0 in range(r_first, n_q, row_block):
        rows = np.arange(r0, min(n_q, r0 + row_block))
        kl[rows], lse1[rows], lse2[rows] = forward_rows(
            Q1, K1, Q2, K2, s1, s2, causal, direction, b, h, rows)
    q1h, q2h = _head(Q1, b, h), _head(Q2, b, h)
    k1c, k2c = _head(K1, b, h)[keys], _head(K2, b, h)[keys]
    g = np.asarray(g, dtype=np.float64).reshape(-1)
    dk1 = np.zeros((keys.size, q1h.shape[1]))
    dk2 = np.zeros((keys.size, q2h.shape[1]))
    for r0 in range(r_first, n_q, row_block):
        rows = np.arange(r0, min(n_q, r0 + row_block))
        mask = allowed_mask(rows, n_q, n_k, causal)[:, keys]
        S1 = s1 * (q1h[rows] @ k1c.T)
        S2 = s2 * (q2h[rows] @ k2c.T)
        with np.errstate(invalid="ignore"):
            logP1 = np.where(mask, S1 - lse1[rows, None], -np.inf)
            logP2 = np.where(mask, S2 - lse2[rows, None], -np.inf)
        qd = dict(mask=mask, P1=np.exp(logP1), P2=np.exp(logP2), logP1=logP1, logP2=logP2)
        dS1, dS2 = _logit_grads(qd, kl[rows], g[rows], direction)
        dk1 += s1 * (dS1.T @ q1h[rows])
        dk2 += s2 * (dS2.T @ q2h[rows])
    return dk1, dk2


def forward(Q1, K1, Q2, K2, s1, s2, causal=False, direction=FWD, row_block=256):
    """KL, LSE1, LSE2 as [B, H, N_Q] fp64 arrays for every row of every head."""
    B, H, n_q = Q1.shape[:3]
    kl = np.empty((B, H, n_q))
    lse1 = np.empty((B, H, n_q))
    lse2 = np.empty((B, H, n_q))
    for b in range(B):
        for h in range(H):
            kl[b, h], lse1[b, h], lse2[b, h] = head_stats_all_rows(
                Q1, K1, Q2, K2, s1, s2, causal, direction, b, h, row_block)
    return kl, lse1, lse2


def backward(Q1, K1, Q2, K2, s1, s2, causal=False, direction=FWD, dkl=None, row_block=256):
    """(kl, lse1, lse2, dQ1, dK1, dQ2, dK2) for every head, fp64.

    dkl: [B, H, N_Q] upstream gradient, None meaning all ones. The gradients
    are those of sum_{b,h,i} dkl[b,h,i] * L[b,h,i].
    """
    _check_direction(direction)
    s1, s2 = _f32(s1), _f32(s2)
    B, H, n_q = Q1.shape[:3]
    if dkl is None:
        dkl = np.ones((B, H, n_q))
    kl = np.empty((B, H, n_q))
    lse1 = np.empty((B, H, n_q))
    lse2 = np.empty((B, H, n_q))
    dQ1 = np.zeros(Q1.shape)
    dQ2 = np.zeros(Q2.shape)
    dK1 = np.zeros(K1.shape)
    dK2 = np.zeros(K2.shape)
    for b in range(B):
        for h in range(H):
            q1h, k1h, q2h, k2h = _head(Q1, b, h), _head(K1, b, h), _head(Q2, b, h), _head(K2, b, h)
            for r0 in range(0, n_q, row_block):
                rows = np.arange(r0, min(n_q, r0 + row_block))
                qd = _rows_quantities(q1h[rows], k1h, q2h[rows], k2h, s1, s2, rows, n_q, causal)
                klr = _row_kl(qd, direction)
                kl[b, h, rows], lse1[b, h, rows], lse2[b, h, rows] = klr, qd["lse1"], qd["lse2"]
                dS1, dS2 = _logit_grads(qd, klr, np.asarray(dkl[b, h, rows], dtype=np.float64), direction)
                dQ1[b, h, rows] = s1 * (dS1 @ k1h)
                dQ2[b, h, rows] = s2 * (dS2 @ k2h)
                dK1[b, h] += s1 * (dS1.T @ q1h[rows])
                dK2[b, h] += s2 * (dS2.T @ q2h[rows])
    return kl, lse1, lse2, dQ1, dK1, dQ2, dK2
