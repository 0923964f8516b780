"""Tile-by-tile evaluation of the online forward (Sec. 3.2) and the split-K merge (Sec. 3.3), in fp64.

TEST INFRASTRUCTURE (see ``oracle/__init__.py``). This is not the oracle:
the oracle is the plain definition in ``kl_oracle``. This model evaluates the
forward the way a one-pass kernel must, from per-row partial states over key
tiles, so that tests can pin the online reformulation itself against the
plain definition:

* eq:kl-final: L = acc / l1 + LSE2 - LSE1 with acc = sum_j e^{S1_j - m1} (S1_j - S2_j);
* eq:acc-invariant: a partial state over any set of keys holds
  m_t = max S_t, l_t = sum e^{S_t - m_t} and acc = sum e^{S1 - m1} (S1 - S2)
  over exactly those keys;
* the merge of Sec. 3.3: two partial states over disjoint key sets combine by
  rescaling to their common maximum. The paper lists only (m1, l1, acc) for a
  partial; LSE2 needs (m2, l2) as well, so a partial here carries all five
  scalars and (m2, l2) merge by the same log-sum-exp rule.

The streaming pass (eq:acc-update) is the left fold of that merge over the key
tiles in order: a tile's state is computed from its definition, then merged
into the running state. The split-K variant merges whole chunks, each the fold
of its own tiles, in any order.

A row with no allowed key in a set has the empty state (m = -inf, l = 0,
acc = 0); merging with an empty state leaves the other unchanged. Direction
REV evaluates KL(P2 || P1) by swapping the roles of the two distributions.
"""
from __future__ import annotations

import numpy as np

from .kl_oracle import FWD, REV, allowed_mask, _f32


def empty_state(n):
    """Partial state of n rows over no keys."""
    return dict(m1=np.full(n, -np.inf), l1=np.zeros(n), m2=np.full(n, -np.inf), l2=np.zeros(n), acc=np.zeros(n))


def tile_state(S1t, S2t, maskt):
    """Partial state (m1, l1, m2, l2, acc) of every row over one set of keys, from its definition.

    S1t, S2t: logits [rows, keys]; maskt: allowed pairs. Rows with no allowed
    key get the empty state.
    """
    any_key = maskt.any(axis=1)
    m1 = np.where(any_key, np.where(maskt, S1t, -np.inf).max(axis=1), -np.inf)
    m2 = np.where(any_key, np.where(maskt, S2t, -np.inf).max(axis=1), -np.inf)
    ref1 = np.where(any_key, m1, 0.0)[:, None]
    ref2 = np.where(any_key, m2, 0.0)[:, None]
    w1 = np.where(maskt, np.exp(np.where(maskt, S1t, 0.0) - ref1), 0.0)
    w2 = np.where(maskt, np.exp(np.where(maskt, S2t, 0.0) - ref2), 0.0)
    gap = np.where(maskt, S1t - S2t, 0.0)
    return dict(m1=m1, l1=w1.sum(axis=1), m2=m2, l2=w2.sum(axis=1), acc=(w1 * gap).sum(axis=1))


def _weight(m_part, m_all):
    """e^{m_part - m_all}, and 0 for an empty part (its sums are 0 anyway)."""
    return np.where(np.isneginf(m_part), 0.0, np.exp(np.where(np.isneginf(m_part), 0.0, m_part - np.where(
        np.isneginf(m_all), 0.0, m_all))))


def merge_states(a, b):
    """Combine two partial states over disjoint key sets (split-K merge, Sec. 3.3)."""
    m1 = np.maximum(a["m1"], b["m1"])
    m2 = np.maximum(a["m2"], b["m2"])
    wa1, wb1 = _weight(a["m1"], m1), _weight(b["m1"], m1)
    wa2, wb2 = _weight(a["m2"], m2), _weight(b["m2"], m2)
    return dict(m1=m1, m2=m2,
                l1=a["l1"] * wa1 + b["l1"] * wb1,
                l2=a["l2"] * wa2 + b["l2"] * wb2,
                acc=a["acc"] * wa1 + b["acc"] * wb1)


def finalize(st):
    """KL, LSE1, LSE2 of complete rows: LSE_t = m_t + ln l_t, KL = acc / l1 + LSE2 - LSE1 (eq:kl-final).

    Rows with no allowed key: KL = 0, LSE = -inf.
    """
    seen = st["l1"] > 0
    with np.errstate(divide="ignore"):
        lse1 = np.where(seen, st["m1"] + np.log(np.where(seen, st["l1"], 1.0)), -np.inf)
        lse2 = np.where(seen, st["m2"] + np.log(np.where(seen, st["l2"], 1.0)), -np.inf)
    gap = np.where(seen, lse2, 0.0) - np.where(seen, lse1, 0.0)
    kl = np.where(seen, st["acc"] / np.where(seen, st["l1"], 1.0) + gap, 0.0)
    return kl, lse1, lse2


def _logits(q1, k1, q2, k2, s1, s2):
    return _f32(s1) * (np.asarray(q1, np.float64) @ np.asarray(k1, np.float64).T), \
        _f32(s2) * (np.asarray(q2, np.float64) @ np.asarray(k2, np.float64).T)


def streamed_state(S1, S2, mask, k_begin, k_end, block_k):
    """Left fold of merge_states over the key tiles [j, j + block_k) of [k_begin, k_end), in key order."""
    st = empty_state(S1.shape[0])
    for j in range(k_begin, k_end, block_k):
        e = min(k_end, j + block_k)
        st = merge_states(st, tile_state(S1[:, j:e], S2[:, j:e], mask[:, j:e]))
    return st


def online_forward_head(q1, k1, q2, k2, s1, s2, causal=False, direction=FWD, block_k=64):
    """KL, LSE1, LSE2 of one head from one streaming pass over key tiles of ``block_k``.

    q1: [N_Q, d1], k1: [N_K, d1], q2: [N_Q, d2], k2: [N_K, d2].
    """
    S1, S2 = _logits(q1, k1, q2, k2, s1, s2)
    n_q, n_k = S1.shape
    mask = allowed_mask(np.arange(n_q), n_q, n_k, causal)
    if direction == REV:
        kl, lse2, lse1 = finalize(streamed_state(S2, S1, mask, 0, n_k, block_k))
        return kl, lse1, lse2
    return finalize(streamed_state(S1, S2, mask, 0, n_k, block_k))


def split_merge_forward_head(q1, k1, q2, k2, s1, s2, causal=False, direction=FWD,
                             splits=4, block_k=64, order=None):
    """KL, LSE1, LSE2 via W = ``splits`` contiguous key chunks merged in ``order``.

    Each chunk is streamed on its own from the empty state; the W chunk states
    are then merged one by one in the given order (a permutation of
    range(W), default ascending).
    """
    S1, S2 = _logits(q1, k1, q2, k2, s1, s2)
    if direction == REV:
        S1, S2 = S2, S1
    n_q, n_k = S1.shape
    mask = allowed_mask(np.arange(n_q), n_q, n_k, causal)
    ck = -(-n_k // splits)
    parts = [streamed_state(S1, S2, mask, w * ck, min(n_k, (w + 1) * ck), block_k) for w in range(splits)]
    order = list(range(splits)) if order is None else list(order)
    st = parts[order[0]]
    for w in order[1:]:
        st = merge_states(st, parts[w])
    kl, la, lb = finalize(st)
    return (kl, lb, la) if direction == REV else (kl, la, lb)
