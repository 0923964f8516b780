"""Algorithm 1 (Sec. 3.2) executed tile by tile in fp64, and the split-K merge (Sec. 3.3).

TEST INFRASTRUCTURE (see ``oracle/__init__.py``). This is not the oracle:
the oracle is the plain definition in ``kl_oracle``. This model takes the
paper's online steps in the paper's order so that tests can pin the online
reformulation itself against the plain definition:

* eq:kl-final: L = acc / l1 + LSE2 - LSE1 with acc = sum_j e^{S1_j - m1} (S1_j - S2_j);
* eq:acc-invariant / eq:acc-update: after each key tile the five per-row
  scalars (m1, l1, m2, l2, acc) equal their definitions over the tiles seen;
* the split-K merge (Sec. 3.3): partial states over contiguous key chunks
  combine by rescaling to their common maximum. The paper lists only
  (m1, l1, acc) for a partial; LSE2 needs (m2, l2) as well, so a partial here
  carries all five scalars and (m2, l2) merge by the same log-sum-exp rule.

Masked entries contribute exactly 0 to l and acc, and a correction factor
between two -inf maxima is taken as 1 (both states are still empty).
Direction REV evaluates KL(P2 || P1) by running the same steps with the roles
of the two distributions swapped.
"""
from __future__ import annotations

import numpy as np

from .kl_oracle import FWD, REV, allowed_mask, _f32


def _exp_diff(a, b):
    """e^{a - b} elementwise, with e^{-inf - (-inf)} taken as 1 (empty state)."""
    with np.errstate(invalid="ignore"):
        d = a - b
    return np.where(np.isneginf(a) & np.isneginf(b), 1.0, np.exp(np.where(np.isnan(d), 0.0, d)))


def _init_state(n):
    return dict(m1=np.full(n, -np.inf), l1=np.zeros(n), m2=np.full(n, -np.inf),
                l2=np.zeros(n), acc=np.zeros(n))


def _update(st, S1t, S2t, maskt):
    """One inner-loop step of Algorithm 1 on a key tile (rows x tile keys)."""
    S1m = np.where(maskt, S1t, -np.inf)
    S2m = np.where(maskt, S2t, -np.inf)
    # update maximums
    m1n = np.maximum(st["m1"], S1m.max(axis=1))
    m2n = np.maximum(st["m2"], S2m.max(axis=1))
    # correction factors
    a1 = _exp_diff(st["m1"], m1n)
    a2 = _exp_diff(st["m2"], m2n)
    # unnormalised probabilities of the tile (0 where masked or the row is still empty)
    with np.errstate(invalid="ignore"):
        P1t = np.where(maskt, np.exp(S1m - np.where(np.isneginf(m1n), 0.0, m1n)[:, None]), 0.0)
        P2t = np.where(maskt, np.exp(S2m - np.where(np.isneginf(m2n), 0.0, m2n)[:, None]), 0.0)
    # running sums and the accumulator
    st["l1"] = a1 * st["l1"] + P1t.sum(axis=1)
    st["l2"] = a2 * st["l2"] + P2t.sum(axis=1)
    diff = np.where(maskt, S1t - S2t, 0.0)
    st["acc"] = a1 * st["acc"] + (P1t * diff).sum(axis=1)
    st["m1"], st["m2"] = m1n, m2n
    return st


def _finalize(st):
    """LSE_t = m_t + log l_t; KL = acc / l1 + LSE2 - LSE1 (eq:kl-final). Empty rows: KL = 0."""
    with np.errstate(divide="ignore", invalid="ignore"):
        lse1 = np.where(st["l1"] > 0, st["m1"] + np.log(st["l1"]), -np.inf)
        lse2 = np.where(st["l2"] > 0, st["m2"] + np.log(st["l2"]), -np.inf)
        kl = np.where(st["l1"] > 0, st["acc"] / np.where(st["l1"] > 0, st["l1"], 1.0) + lse2 - lse1, 0.0)
    return kl, lse1, lse2


def _logits(q1, k1, q2, k2, s1, s2):
    return _f32(s1) * (np.asarray(q1, np.float64) @ np.asarray(k1, np.float64).T), \
        _f32(s2) * (np.asarray(q2, np.float64) @ np.asarray(k2, np.float64).T)


def _chunk_state(S1, S2, mask, k0, k1_, block_k):
    st = _init_state(S1.shape[0])
    for j0 in range(k0, k1_, block_k):
        j1 = min(k1_, j0 + block_k)
        st = _update(st, S1[:, j0:j1], S2[:, j0:j1], mask[:, j0:j1])
    return st


def online_forward_head(q1, k1, q2, k2, s1, s2, causal=False, direction=FWD, block_k=64):
    """KL, LSE1, LSE2 of one head via Algorithm 1 with key tiles of ``block_k``.

    q1: [N_Q, d1], k1: [N_K, d1], q2: [N_Q, d2], k2: [N_K, d2].
    """
    S1, S2 = _logits(q1, k1, q2, k2, s1, s2)
    n_q, n_k = S1.shape
    mask = allowed_mask(np.arange(n_q), n_q, n_k, causal)
    if direction == REV:
        kl, lse2, lse1 = _finalize(_chunk_state(S2, S1, mask, 0, n_k, block_k))
        return kl, lse1, lse2
    return _finalize(_chunk_state(S1, S2, mask, 0, n_k, block_k))


def merge_states(a, b):
    """Combine two partial states over disjoint key sets (split-K merge, Sec. 3.3)."""
    m1 = np.maximum(a["m1"], b["m1"])
    m2 = np.maximum(a["m2"], b["m2"])
    ea1, eb1 = _exp_diff(a["m1"], m1), _exp_diff(b["m1"], m1)
    ea2, eb2 = _exp_diff(a["m2"], m2), _exp_diff(b["m2"], m2)
    return dict(m1=m1, m2=m2,
                l1=a["l1"] * ea1 + b["l1"] * eb1,
                l2=a["l2"] * ea2 + b["l2"] * eb2,
                acc=a["acc"] * ea1 + b["acc"] * eb1)


def split_merge_forward_head(q1, k1, q2, k2, s1, s2, causal=False, direction=FWD,
                             splits=4, block_k=64, order=None):
    """KL, LSE1, LSE2 via W = ``splits`` contiguous key chunks merged in ``order``.

    Each chunk runs Algorithm 1 from the initial state on its own keys; the W
    partial states are then merged one by one in the given order (a
    permutation of range(W), default ascending).
    """
    S1, S2 = _logits(q1, k1, q2, k2, s1, s2)
    if direction == REV:
        S1, S2 = S2, S1
    n_q, n_k = S1.shape
    mask = allowed_mask(np.arange(n_q), n_q, n_k, causal)
    ck = -(-n_k // splits)
    parts = [_chunk_state(S1, S2, mask, w * ck, min(n_k, (w + 1) * ck), block_k) for w in range(splits)]
    order = list(range(splits)) if order is None else list(order)
    st = parts[order[0]]
    for w in order[1:]:
        st = merge_states(st, parts[w])
    kl, la, lb = _finalize(st)
    return (kl, lb, la) if direction == REV else (kl, la, lb)
