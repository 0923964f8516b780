"""Pins of the sigmoid-score oracle (oracle/sigmoid_oracle.py) to facts that do
not come from the oracle itself: scipy's independent kl_div / expit, a value
worked by hand, the softmax oracle's eq:kl-def (the divergence reduces to it
for normalised rows), exact zeros for identical inputs, torch fp64 autograd,
central finite differences and a pure-Python brute force of the masking."""
import math

import numpy as np
import pytest
import scipy.special

import oracle
from oracle import sigmoid_oracle as so
from oracle.kl_oracle import FWD, REV, allowed_mask
from paper_2606_20005_amd import inputs


def _case(n_q=40, n_k=70, d1=16, d2=8, seed=3, B=1, H=2):
    rng = np.random.default_rng(seed)
    Q1, K1 = rng.standard_normal((B, H, n_q, d1)), rng.standard_normal((B, H, n_k, d1))
    Q2, K2 = rng.standard_normal((B, H, n_q, d2)), rng.standard_normal((B, H, n_k, d2))
    return Q1, K1, Q2, K2


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("direction", [FWD, REV])
def test_matches_scipy_kl_div(causal, direction):
    """scipy.special.kl_div(x, y) = x log(x/y) - x + y elementwise, expit = sigmoid."""
    Q1, K1, Q2, K2 = _case()
    s1, s2 = 0.25, 0.5
    L, M1, M2 = so.forward(Q1, K1, Q2, K2, s1, s2, causal, direction)
    for b, h in ((0, 0), (0, 1)):
        S1 = s1 * Q1[b, h] @ K1[b, h].T
        S2 = s2 * Q2[b, h] @ K2[b, h].T
        mask = allowed_mask(np.arange(Q1.shape[2]), Q1.shape[2], K1.shape[2], causal)
        A1, A2 = scipy.special.expit(S1), scipy.special.expit(S2)
        x, y = (A1, A2) if direction == FWD else (A2, A1)
        ref = np.where(mask, scipy.special.kl_div(x, y), 0.0).sum(axis=1)
        np.testing.assert_allclose(L[b, h], ref, rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(M1[b, h], np.where(mask, A1, 0).sum(axis=1), rtol=1e-13)
        np.testing.assert_allclose(M2[b, h], np.where(mask, A2, 0).sum(axis=1), rtol=1e-13)


def test_hand_worked_single_key():
    """One key, d = 1: S1 = 0 gives A1 = 1/2, S2 = ln 3 gives A2 = 3/4.
    FWD: 1/2 ln(2/3) - 1/2 + 3/4 = 0.0472674459459178...
    REV: 3/4 ln(3/2) - 3/4 + 1/2 = 0.0540988310811233..."""
    Q1, K1 = np.zeros((1, 1, 1, 1)), np.ones((1, 1, 1, 1))
    Q2, K2 = np.full((1, 1, 1, 1), math.log(3.0)), np.ones((1, 1, 1, 1))
    L, M1, M2 = so.forward(Q1, K1, Q2, K2, 1.0, 1.0, False, FWD)
    assert abs(L[0, 0, 0] - 0.0472674459459178) < 1e-15
    assert abs(M1[0, 0, 0] - 0.5) < 1e-16 and abs(M2[0, 0, 0] - 0.75) < 1e-15
    L, _, _ = so.forward(Q1, K1, Q2, K2, 1.0, 1.0, False, REV)
    assert abs(L[0, 0, 0] - 0.0540988310811233) < 1e-15


def test_row_value_reduces_to_eq_kl_def_for_normalised_rows():
    """Fed softmax probabilities instead of sigmoid scores, the row value of
    the generalized divergence is eq:kl-def (the -P1 + P2 terms cancel)."""
    d = inputs.make("tiny", n_q=50, n_k=90)
    w = d["w"]
    kl, _, _ = oracle.forward(d["Q1"], d["K1"], d["Q2"], d["K2"], w.s1, w.s2, True, FWD)
    from oracle import kl_oracle
    q1, k1, q2, k2 = (d[k][0, 0].astype(np.float64) for k in ("Q1", "K1", "Q2", "K2"))
    rows = np.arange(50)
    qd = kl_oracle._rows_quantities(q1, k1, q2, k2, np.float32(w.s1), np.float32(w.s2), rows, 50, True)
    rd = dict(mask=qd["mask"], A1=qd["P1"], A2=qd["P2"], lA1=np.where(qd["mask"], qd["logP1"], 0.0),
              lA2=np.where(qd["mask"], qd["logP2"], 0.0))
    L, M1, M2 = so._row_values(rd, FWD)
    np.testing.assert_allclose(L, kl[0, 0], rtol=1e-10, atol=1e-13)
    np.testing.assert_allclose(M1, 1.0, rtol=1e-13)
    # and the stand-alone helper on two normalised two-point distributions
    assert abs(so.generalized_kl([0.2, 0.8], [0.5, 0.5]) - (0.2 * math.log(0.4) + 0.8 * math.log(1.6))) < 1e-15


@pytest.mark.parametrize("causal", [False, True])
def test_identical_inputs_give_exact_zeros(causal):
    Q1, K1, _, _ = _case(d2=16)
    out = so.backward(Q1, K1, Q1, K1, 0.3, 0.3, causal, FWD)
    assert np.all(out[0] == 0.0)
    for gr in out[3:]:
        assert np.all(gr == 0.0)


@pytest.mark.parametrize("causal", [False, True])
def test_nonnegative_and_rev_swaps_roles(causal):
    Q1, K1, Q2, K2 = _case(seed=8)
    L, M1, M2 = so.forward(Q1, K1, Q2, K2, 0.4, 0.7, causal, FWD)
    assert L.min() >= -1e-13
    Lr, M1r, M2r = so.forward(Q1, K1, Q2, K2, 0.4, 0.7, causal, REV)
    Ls, M2s, M1s = so.forward(Q2, K2, Q1, K1, 0.7, 0.4, causal, FWD)
    np.testing.assert_allclose(Lr, Ls, rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(M1r, M1s, rtol=1e-14)


def test_causal_masking_brute_force():
    """Pure-Python sums over the allowed keys (bottom-right alignment), N_Q < N_K and N_Q > N_K."""
    for n_q, n_k in ((6, 9), (9, 6)):
        Q1, K1, Q2, K2 = _case(n_q=n_q, n_k=n_k, d1=3, d2=2, H=1, seed=n_q)
        L, M1, M2 = so.forward(Q1, K1, Q2, K2, 0.5, 0.5, True, FWD)
        for i in range(n_q):
            tot, m1, m2 = 0.0, 0.0, 0.0
            for j in range(n_k):
                if j > n_k - n_q + i:
                    continue
                s1 = 0.5 * sum(Q1[0, 0, i, c] * K1[0, 0, j, c] for c in range(3))
                s2 = 0.5 * sum(Q2[0, 0, i, c] * K2[0, 0, j, c] for c in range(2))
                a1, a2 = 1 / (1 + math.exp(-s1)), 1 / (1 + math.exp(-s2))
                tot += a1 * math.log(a1 / a2) - a1 + a2
                m1 += a1
                m2 += a2
            assert abs(L[0, 0, i] - tot) < 1e-12 and abs(M1[0, 0, i] - m1) < 1e-12 and abs(M2[0, 0, i] - m2) < 1e-12


def _torch_grads(Q1, K1, Q2, K2, s1, s2, causal, direction, g):
    import torch
    t = [torch.tensor(x, dtype=torch.float64, requires_grad=True) for x in (Q1, K1, Q2, K2)]
    n_q, n_k = Q1.shape[2], K1.shape[2]
    mask = torch.tensor(allowed_mask(np.arange(n_q), n_q, n_k, causal))
    S1 = float(np.float32(s1)) * t[0] @ t[1].transpose(-1, -2)
    S2 = float(np.float32(s2)) * t[2] @ t[3].transpose(-1, -2)
    la, lb = torch.nn.functional.logsigmoid(S1), torch.nn.functional.logsigmoid(S2)
    if direction == REV:
        la, lb = lb, la
    term = torch.exp(la) * (la - lb) - torch.exp(la) + torch.exp(lb)
    L = torch.where(mask, term, torch.zeros_like(term)).sum(-1)
    (L * torch.tensor(g)).sum().backward()
    return [x.grad.numpy() for x in t]


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("direction", [FWD, REV])
def test_gradients_match_torch_autograd(causal, direction):
    Q1, K1, Q2, K2 = _case(seed=11)
    g = np.random.default_rng(2).uniform(-1.5, 1.5, Q1.shape[:3])
    out = so.backward(Q1, K1, Q2, K2, 0.3, 0.6, causal, direction, g)
    ref = _torch_grads(Q1, K1, Q2, K2, 0.3, 0.6, causal, direction, g)
    for got, r in zip((out[3], out[4], out[5], out[6]), ref):
        np.testing.assert_allclose(got, r, rtol=1e-10, atol=1e-12)


def test_central_finite_differences():
    Q1, K1, Q2, K2 = _case(n_q=12, n_k=20, d1=6, d2=4, H=1, seed=21)
    g = np.random.default_rng(4).uniform(0.5, 1.5, Q1.shape[:3])
    s1, s2 = 0.5, 0.75
    out = so.backward(Q1, K1, Q2, K2, s1, s2, True, FWD, g)
    grads = {0: out[3], 1: out[4], 2: out[5], 3: out[6]}
    rng = np.random.default_rng(9)
    h = 1e-5
    for idx in range(4):
        X = [Q1, K1, Q2, K2]
        for _ in range(4):
            v = rng.standard_normal(X[idx].shape)
            Xp = [x.copy() for x in X]
            Xm = [x.copy() for x in X]
            Xp[idx] += h * v
            Xm[idx] -= h * v
            fp = (so.forward(*Xp, s1, s2, True, FWD)[0] * g).sum()
            fm = (so.forward(*Xm, s1, s2, True, FWD)[0] * g).sum()
            num = (fp - fm) / (2 * h)
            ana = (grads[idx] * v).sum()
            assert abs(num - ana) <= 1e-6 * max(1.0, abs(ana)), (idx, num, ana)


def test_empty_rows():
    """Causal with N_Q > N_K: the first rows see no key: L = 0, masses 0, zero gradients."""
    Q1, K1, Q2, K2 = _case(n_q=10, n_k=4, seed=5, H=1)
    out = so.backward(Q1, K1, Q2, K2, 0.5, 0.5, True, FWD)
    assert np.all(out[0][0, 0, :6] == 0) and np.all(out[1][0, 0, :6] == 0) and np.all(out[2][0, 0, :6] == 0)
    assert np.all(out[3][0, 0, :6] == 0) and np.all(out[5][0, 0, :6] == 0)


def test_dq_dk_rows_agree_with_full_backward():
    Q1, K1, Q2, K2 = _case(seed=13)
    g = np.random.default_rng(6).uniform(0.5, 1.5, Q1.shape[:3])
    out = so.backward(Q1, K1, Q2, K2, 0.3, 0.6, True, REV, g)
    rows = np.array([0, 5, 39])
    q1, q2 = so.dq_rows(Q1, K1, Q2, K2, 0.3, 0.6, True, REV, 0, 1, rows, g[0, 1, rows])
    np.testing.assert_allclose(q1, out[3][0, 1, rows], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(q2, out[5][0, 1, rows], rtol=1e-12, atol=1e-14)
    keys = np.array([0, 33, 69])
    k1, k2 = so.dk_rows(Q1, K1, Q2, K2, 0.3, 0.6, True, REV, 0, 1, keys, g[0, 1], row_block=16)
    np.testing.assert_allclose(k1, out[4][0, 1, keys], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(k2, out[6][0, 1, keys], rtol=1e-12, atol=1e-14)
