"""Pins of the fp64 oracle against facts fixed by the paper and by mathematics.

None of these re-types the oracle's formulas: each compares it with an
independent fact (a closed form, a library routine computing the same
quantity by another route, an identity, finite differences of the forward
definition, or the exact zero of identical distributions). A plausible
mistake in the oracle (a dropped term, a wrong sign or index, a transposed
operand, the wrong causal alignment, a missing scale) fails at least one.
"""
import math

import numpy as np
import pytest
import scipy.special as sps

import oracle
from oracle.kl_oracle import FWD, REV
from paper_2606_20005_amd import inputs


def _rand_case(B=1, H=2, n_q=7, n_k=11, d1=5, d2=3, seed=0, scale=1.0):
    rng = np.random.default_rng(seed)
    Q1 = scale * rng.standard_normal((B, H, n_q, d1))
    K1 = scale * rng.standard_normal((B, H, n_k, d1))
    Q2 = scale * rng.standard_normal((B, H, n_q, d2))
    K2 = scale * rng.standard_normal((B, H, n_k, d2))
    return Q1, K1, Q2, K2


def _f32(x):
    return float(np.float32(x))


# --------------------------------------------------------------- forward pins

@pytest.mark.parametrize("causal", [False, True])
def test_identical_inputs_give_exact_zero(causal):
    """(Q2,K2,s2) = (Q1,K1,s1) => P1 = P2 => KL = 0 and every gradient = 0 exactly."""
    d = inputs.make("tiny", "identical")
    w = d["w"]
    kl, l1, l2, dQ1, dK1, dQ2, dK2 = oracle.backward(d["Q1"], d["K1"], d["Q2"], d["K2"], w.s1, w.s2,
                                                     causal, FWD, d["g"])
    assert np.all(kl == 0.0)
    assert np.array_equal(l1, l2)
    for G in (dQ1, dK1, dQ2, dK2):
        assert np.all(G == 0.0)


@pytest.mark.parametrize("direction", [FWD, REV])
@pytest.mark.parametrize("causal", [False, True])
def test_gibbs_nonnegative(causal, direction):
    Q1, K1, Q2, K2 = _rand_case(H=3, n_q=40, n_k=40, d1=16, d2=8, seed=1, scale=1.5)
    kl, _, _ = oracle.forward(Q1, K1, Q2, K2, 0.5, 0.7, causal, direction)
    assert kl.min() >= -1e-12
    assert kl.max() > 0.01


def test_matches_scipy_logsoftmax_definition():
    """Non-causal KL and LSE against scipy's logsumexp / kl_div / rel_entr (library route)."""
    Q1, K1, Q2, K2 = _rand_case(H=2, n_q=9, n_k=13, d1=6, d2=4, seed=2)
    s1, s2 = 0.37, 1.3
    kl, lse1, lse2 = oracle.forward(Q1, K1, Q2, K2, s1, s2, False, FWD)
    klr, _, _ = oracle.forward(Q1, K1, Q2, K2, s1, s2, False, REV)
    for h in range(2):
        S1 = _f32(s1) * Q1[0, h] @ K1[0, h].T
        S2 = _f32(s2) * Q2[0, h] @ K2[0, h].T
        np.testing.assert_allclose(lse1[0, h], sps.logsumexp(S1, axis=1), rtol=1e-14)
        np.testing.assert_allclose(lse2[0, h], sps.logsumexp(S2, axis=1), rtol=1e-14)
        P1, P2 = sps.softmax(S1, axis=1), sps.softmax(S2, axis=1)
        np.testing.assert_allclose(kl[0, h], sps.rel_entr(P1, P2).sum(axis=1), rtol=1e-11, atol=1e-14)
        np.testing.assert_allclose(klr[0, h], sps.rel_entr(P2, P1).sum(axis=1), rtol=1e-11, atol=1e-14)


def test_q1_zero_uniform_closed_form():
    """Q1 = 0 => P1 uniform over the n_i allowed keys: LSE1 = ln n_i and
    KL_i = -ln n_i - (1/n_i) sum_j log P2_j (log P2 via scipy's log_softmax)."""
    for causal in (False, True):
        d = inputs.make("tiny", "q1zero", n_q=64, n_k=96, causal=causal)
        w = d["w"]
        kl, lse1, lse2 = oracle.forward(d["Q1"], d["K1"], d["Q2"], d["K2"], w.s1, w.s2, causal, FWD)
        S2 = _f32(w.s2) * d["Q2"][0, 0].astype(np.float64) @ d["K2"][0, 0].astype(np.float64).T
        for i in range(w.n_q):
            n = (w.n_k - w.n_q + i + 1) if causal else w.n_k
            logp2 = sps.log_softmax(S2[i, :n])
            assert abs(lse1[0, 0, i] - math.log(n)) <= 1e-12 * math.log(n)
            ref = -math.log(n) - logp2.mean()
            assert abs(kl[0, 0, i] - ref) <= 1e-12 * abs(ref)


def test_q2_zero_entropy_closed_form():
    """Q2 = 0 => P2 uniform: KL_i = ln n - H(P1) with H from scipy.stats.entropy."""
    from scipy.stats import entropy
    Q1, K1, Q2, K2 = _rand_case(H=1, n_q=12, n_k=30, d1=8, d2=4, seed=3)
    Q2[:] = 0
    for causal in (False, True):
        kl, _, _ = oracle.forward(Q1, K1, Q2, K2, 0.8, 0.5, causal, FWD)
        S1 = _f32(0.8) * Q1[0, 0] @ K1[0, 0].T
        for i in range(12):
            n = (30 - 12 + i + 1) if causal else 30
            ref = math.log(n) - entropy(sps.softmax(S1[i, :n]))
            assert abs(kl[0, 0, i] - ref) <= 1e-12 * max(1.0, abs(ref))


def test_two_keys_bernoulli_closed_form():
    """N_K = 2 => KL of two Bernoulli distributions with p = sigmoid(S1_0 - S1_1)."""
    Q1, K1, Q2, K2 = _rand_case(H=2, n_q=6, n_k=2, d1=4, d2=3, seed=4, scale=2.0)
    s1, s2 = 0.6, 0.9
    for direction in (FWD, REV):
        kl, _, _ = oracle.forward(Q1, K1, Q2, K2, s1, s2, False, direction)
        for h in range(2):
            S1 = _f32(s1) * Q1[0, h] @ K1[0, h].T
            S2 = _f32(s2) * Q2[0, h] @ K2[0, h].T
            p = 1 / (1 + np.exp(-(S1[:, 0] - S1[:, 1])))
            q = 1 / (1 + np.exp(-(S2[:, 0] - S2[:, 1])))
            if direction == REV:
                p, q = q, p
            ref = p * np.log(p / q) + (1 - p) * np.log((1 - p) / (1 - q))
            np.testing.assert_allclose(kl[0, h], ref, rtol=1e-12, atol=1e-15)


def test_hand_worked_example():
    """A worked example by hand: q1 = 1, K1 = [[1],[0]], s1 = 1 gives S1 = [1, 0],
    P1 = (e/(e+1), 1/(e+1)); q2 = 0 gives P2 = (1/2, 1/2); so
    KL = ln 2 - H(P1) = ln 2 + p ln p + (1-p) ln(1-p) with p = e/(1+e)."""
    Q1 = np.array([[[[1.0]]]]); K1 = np.array([[[[1.0], [0.0]]]])
    Q2 = np.array([[[[0.0]]]]); K2 = np.array([[[[3.0], [-2.0]]]])
    kl, lse1, lse2 = oracle.forward(Q1, K1, Q2, K2, 1.0, 1.0, False, FWD)
    p = math.e / (1 + math.e)
    assert abs(kl[0, 0, 0] - (math.log(2) + p * math.log(p) + (1 - p) * math.log(1 - p))) < 1e-15
    assert abs(lse1[0, 0, 0] - math.log(math.e + 1)) < 1e-15
    assert abs(lse2[0, 0, 0] - math.log(2)) < 1e-15


def test_causal_bottom_right_alignment():
    """Causal with N_Q <= N_K: row i sees exactly keys 0 .. N_K - N_Q + i.
    Checked by brute force: each row equals the non-causal value computed on
    the truncated key set. For N_Q = N_K row 0 has one key: KL = 0, LSE = S[0,0]."""
    Q1, K1, Q2, K2 = _rand_case(H=1, n_q=5, n_k=9, d1=4, d2=4, seed=5)
    kl, lse1, lse2 = oracle.forward(Q1, K1, Q2, K2, 0.7, 0.4, True, FWD)
    for i in range(5):
        n = 9 - 5 + i + 1
        k, a, b = oracle.forward(Q1[:, :, i:i + 1], K1[:, :, :n], Q2[:, :, i:i + 1], K2[:, :, :n],
                                 0.7, 0.4, False, FWD)
        assert abs(k[0, 0, 0] - kl[0, 0, i]) < 1e-13
        assert abs(a[0, 0, 0] - lse1[0, 0, i]) < 1e-13
    Q1, K1, Q2, K2 = _rand_case(H=1, n_q=6, n_k=6, d1=4, d2=4, seed=6)
    kl, lse1, _ = oracle.forward(Q1, K1, Q2, K2, 0.7, 0.4, True, FWD)
    assert kl[0, 0, 0] == 0.0
    assert lse1[0, 0, 0] == _f32(0.7) * float(Q1[0, 0, 0] @ K1[0, 0, 0])
    _, _, _, dQ1, dK1, dQ2, dK2 = oracle.backward(Q1[:, :, :1], K1, Q2[:, :, :1], K2, 0.7, 0.4,
                                                  True, FWD)  # row 0 alone: N_Q=1 shifts alignment
    # a lone query row sees all 6 keys under bottom-right alignment
    k_all, _, _ = oracle.forward(Q1[:, :, :1], K1, Q2[:, :, :1], K2, 0.7, 0.4, False, FWD)
    k_c, _, _ = oracle.forward(Q1[:, :, :1], K1, Q2[:, :, :1], K2, 0.7, 0.4, True, FWD)
    assert k_all[0, 0, 0] == k_c[0, 0, 0]


def test_empty_rows_when_more_queries_than_keys():
    Q1, K1, Q2, K2 = _rand_case(H=1, n_q=6, n_k=4, d1=3, d2=3, seed=7)
    kl, lse1, lse2, dQ1, dK1, dQ2, dK2 = oracle.backward(Q1, K1, Q2, K2, 1.0, 1.0, True, FWD)
    assert np.all(kl[0, 0, :2] == 0) and np.all(np.isneginf(lse1[0, 0, :2])) and np.all(np.isneginf(lse2[0, 0, :2]))
    assert np.all(dQ1[0, 0, :2] == 0) and np.all(dQ2[0, 0, :2] == 0)
    assert np.all(np.isfinite(kl)) and np.all(np.isfinite(dK1)) and np.all(np.isfinite(dK2))
    assert kl[0, 0, 2] == 0.0   # first non-empty row sees one key


def test_jeffreys_identity_and_rev_swap():
    """KL(P1||P2) + KL(P2||P1) = sum_j (P1 - P2)(S1 - S2);  REV(1,2) = FWD(2,1)."""
    Q1, K1, Q2, K2 = _rand_case(H=2, n_q=8, n_k=10, d1=5, d2=7, seed=8)
    s1, s2 = 0.45, 0.8
    for causal in (False, True):
        kf, a1, a2 = oracle.forward(Q1, K1, Q2, K2, s1, s2, causal, FWD)
        kr, b1, b2 = oracle.forward(Q1, K1, Q2, K2, s1, s2, causal, REV)
        ks, c1, c2 = oracle.forward(Q2, K2, Q1, K1, s2, s1, causal, FWD)
        np.testing.assert_allclose(kr, ks, rtol=0, atol=1e-15)
        np.testing.assert_array_equal(b1, c2)
        np.testing.assert_array_equal(a1, b1)
        for h in range(2):
            S1 = _f32(s1) * Q1[0, h] @ K1[0, h].T
            S2 = _f32(s2) * Q2[0, h] @ K2[0, h].T
            m = oracle.allowed_mask(np.arange(8), 8, 10, causal)
            S1m, S2m = np.where(m, S1, -np.inf), np.where(m, S2, -np.inf)
            P1, P2 = sps.softmax(S1m, axis=1), sps.softmax(S2m, axis=1)
            ref = np.where(m, (P1 - P2) * (S1 - S2), 0).sum(axis=1)
            np.testing.assert_allclose(kf[0, h] + kr[0, h], ref, rtol=1e-12, atol=1e-14)


def test_key_shift_invariance():
    """K1[j] += v for all j: KL unchanged, LSE1_i += s1 <Q1_i, v>."""
    Q1, K1, Q2, K2 = _rand_case(H=1, n_q=10, n_k=12, d1=6, d2=4, seed=9)
    v = np.random.default_rng(10).standard_normal(6)
    for causal in (False, True):
        kl, l1, _ = oracle.forward(Q1, K1, Q2, K2, 0.6, 0.9, causal, FWD)
        kl2, l1b, _ = oracle.forward(Q1, K1 + v, Q2, K2, 0.6, 0.9, causal, FWD)
        np.testing.assert_allclose(kl2, kl, rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(l1b - l1, _f32(0.6) * (Q1 @ v), rtol=1e-11, atol=1e-12)


# -------------------------------------------------------------- backward pins

@pytest.mark.parametrize("direction", [FWD, REV])
@pytest.mark.parametrize("causal", [False, True])
def test_logit_grad_rows_sum_to_zero(causal, direction):
    Q1, K1, Q2, K2 = _rand_case(H=1, n_q=16, n_k=20, d1=6, d2=5, seed=11, scale=1.3)
    g = np.random.default_rng(12).uniform(0.5, 1.5, 16)
    dS1, dS2, _ = oracle.logit_grads_rows(Q1, K1, Q2, K2, 0.9, 0.6, causal, direction, 0, 0,
                                          np.arange(16), g)
    assert np.abs(dS1.sum(axis=1)).max() <= 1e-12
    assert np.abs(dS2.sum(axis=1)).max() <= 1e-12
    assert np.abs(dS1).max() > 1e-3 and np.abs(dS2).max() > 1e-3


def _loss(Q1, K1, Q2, K2, s1, s2, causal, direction, g):
    kl, _, _ = oracle.forward(Q1, K1, Q2, K2, s1, s2, causal, direction)
    return float((g * kl).sum())


@pytest.mark.parametrize("direction", [FWD, REV])
@pytest.mark.parametrize("causal", [False, True])
def test_grads_match_torch_autograd(causal, direction):
    """Every gradient against torch fp64 CPU autograd of log_softmax-based KL (library route)."""
    import torch
    Q1, K1, Q2, K2 = _rand_case(B=1, H=2, n_q=12, n_k=15, d1=6, d2=4, seed=13)
    g = np.random.default_rng(14).uniform(0.5, 1.5, (1, 2, 12))
    s1, s2 = 0.55, 0.85
    _, _, _, dQ1, dK1, dQ2, dK2 = oracle.backward(Q1, K1, Q2, K2, s1, s2, causal, direction, g)
    T = [torch.tensor(x, requires_grad=True) for x in (Q1, K1, Q2, K2)]
    S1 = _f32(s1) * T[0] @ T[1].transpose(-1, -2)
    S2 = _f32(s2) * T[2] @ T[3].transpose(-1, -2)
    if causal:
        m = torch.tensor(oracle.allowed_mask(np.arange(12), 12, 15, True))
        # a finite fill whose exponential underflows to exactly 0 in fp64 keeps autograd NaN-free
        S1 = S1.masked_fill(~m, -1e4)
        S2 = S2.masked_fill(~m, -1e4)
    a, b = (S1, S2) if direction == FWD else (S2, S1)
    la, lb = torch.log_softmax(a, -1), torch.log_softmax(b, -1)
    terms = la.exp() * (la - lb)
    loss = (torch.tensor(g) * terms.sum(-1)).sum()
    loss.backward()
    for mine, t in zip((dQ1, dK1, dQ2, dK2), T):
        np.testing.assert_allclose(mine, t.grad.numpy(), rtol=1e-10, atol=1e-13)


@pytest.mark.parametrize("direction", [FWD, REV])
def test_tiny_central_finite_differences(direction):
    """Tiny workload (N=256, d=64): loss sum_i g_i KL_i, central differences, h = 1e-5.
    (i) 8 random directional derivatives per tensor; (ii) 256 random entries per tensor."""
    d = inputs.make("tiny")
    w = d["w"]
    Q1, K1, Q2, K2 = (d[k].astype(np.float64) for k in ("Q1", "K1", "Q2", "K2"))
    g = d["g"].astype(np.float64)
    _, _, _, dQ1, dK1, dQ2, dK2 = oracle.backward(Q1, K1, Q2, K2, w.s1, w.s2, False, direction, g)
    grads = (dQ1, dK1, dQ2, dK2)
    rng = np.random.default_rng(15)
    h = 1e-5

    def loss_with(idx, X):
        args = [Q1, K1, Q2, K2]
        args[idx] = X
        return _loss(*args, w.s1, w.s2, False, direction, g)

    for idx, X in enumerate((Q1, K1, Q2, K2)):
        for _ in range(8):
            v = rng.standard_normal(X.shape)
            fd = (loss_with(idx, X + h * v) - loss_with(idx, X - h * v)) / (2 * h)
            an = float((grads[idx] * v).sum())
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (idx, fd, an)
        flat = rng.choice(X.size, 256, replace=False)
        errs = []
        for f in flat:
            e = np.zeros(X.size)
            e[f] = h
            e = e.reshape(X.shape)
            fd = (loss_with(idx, X + e) - loss_with(idx, X - e)) / (2 * h)
            an = grads[idx].reshape(-1)[f]
            errs.append(abs(fd - an) / max(1e-3, abs(an)))
        assert max(errs) <= 1e-5, (idx, max(errs))


def test_dq_dk_rows_match_full_backward():
    """The sampled-row helpers used at full size agree with the full backward."""
    Q1, K1, Q2, K2 = _rand_case(B=1, H=2, n_q=20, n_k=24, d1=5, d2=3, seed=16)
    g = np.random.default_rng(17).uniform(0.5, 1.5, (1, 2, 20))
    for causal in (False, True):
        for direction in (FWD, REV):
            _, _, _, dQ1, dK1, dQ2, dK2 = oracle.backward(Q1, K1, Q2, K2, 0.7, 0.3, causal, direction, g,
                                                          row_block=7)
            rows = np.array([0, 5, 19])
            a, b = oracle.dq_rows(Q1, K1, Q2, K2, 0.7, 0.3, causal, direction, 0, 1, rows, g[0, 1, rows])
            np.testing.assert_allclose(a, dQ1[0, 1, rows], rtol=1e-12, atol=1e-14)
            np.testing.assert_allclose(b, dQ2[0, 1, rows], rtol=1e-12, atol=1e-14)
            keys = np.array([0, 3, 23])
            a, b = oracle.dk_rows(Q1, K1, Q2, K2, 0.7, 0.3, causal, direction, 0, 1, keys, g[0, 1], row_block=6)
            np.testing.assert_allclose(a, dK1[0, 1, keys], rtol=1e-12, atol=1e-14)
            np.testing.assert_allclose(b, dK2[0, 1, keys], rtol=1e-12, atol=1e-14)
            # tail keys: under the causal mask only the last rows are formed
            tail = np.array([17, 21, 23])
            a, b = oracle.dk_rows(Q1, K1, Q2, K2, 0.7, 0.3, causal, direction, 0, 1, tail, g[0, 1], row_block=6)
            np.testing.assert_allclose(a, dK1[0, 1, tail], rtol=1e-12, atol=1e-14)
            np.testing.assert_allclose(b, dK2[0, 1, tail], rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("n_q,n_k", [(24, 10), (10, 24)])
def test_dk_rows_tail_keys_unequal_lengths(n_q, n_k):
    """Sampled dK of tail keys (rows skipped by the causal mask) equals the full
    backward, with more queries than keys (empty rows) and fewer."""
    Q1, K1, Q2, K2 = _rand_case(B=1, H=1, n_q=n_q, n_k=n_k, d1=4, d2=6, seed=18)
    g = np.random.default_rng(19).uniform(0.5, 1.5, (1, 1, n_q))
    _, _, _, _, dK1, _, dK2 = oracle.backward(Q1, K1, Q2, K2, 0.5, 0.9, True, FWD, g, row_block=5)
    for keys in (np.array([n_k - 1]), np.array([n_k - 3, n_k - 2]), np.arange(n_k)):
        a, b = oracle.dk_rows(Q1, K1, Q2, K2, 0.5, 0.9, True, FWD, 0, 0, keys, g[0, 0], row_block=4)
        np.testing.assert_allclose(a, dK1[0, 0, keys], rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(b, dK2[0, 0, keys], rtol=1e-12, atol=1e-14)


def test_scale_invariance_identity_of_gradients():
    """Scaling Q_t by c and K_t by 1/c leaves L unchanged, so <dQ_t, Q_t> = <dK_t, K_t>;
    and rows of dS summing to zero give sum_j dK_t[j] = 0."""
    Q1, K1, Q2, K2 = _rand_case(B=1, H=1, n_q=14, n_k=18, d1=5, d2=4, seed=18)
    for causal in (False, True):
        _, _, _, dQ1, dK1, dQ2, dK2 = oracle.backward(Q1, K1, Q2, K2, 0.9, 0.5, causal, FWD)
        assert abs((dQ1 * Q1).sum() - (dK1 * K1).sum()) < 1e-12
        assert abs((dQ2 * Q2).sum() - (dK2 * K2).sum()) < 1e-12
        assert np.abs(dK1.sum(axis=2)).max() < 1e-12 and np.abs(dK2.sum(axis=2)).max() < 1e-12


# --------------------------------------------------------- online derivation

@pytest.mark.parametrize("direction", [FWD, REV])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("block_k", [1, 7, 64, 256])
def test_online_model_equals_plain_definition(block_k, causal, direction):
    """Algorithm 1 (eq:kl-final with the rescaled accumulator) equals eq:kl-def."""
    d = inputs.make("tiny", n_q=96, n_k=200)
    w = d["w"]
    q1, k1, q2, k2 = (d[k][0, 0].astype(np.float64) for k in ("Q1", "K1", "Q2", "K2"))
    kl, l1, l2 = oracle.online_forward_head(q1, k1, q2, k2, w.s1, w.s2, causal, direction, block_k)
    rk, r1, r2 = oracle.forward(d["Q1"], d["K1"], d["Q2"], d["K2"], w.s1, w.s2, causal, direction)
    np.testing.assert_allclose(kl, rk[0, 0], rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(l1, r1[0, 0], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(l2, r2[0, 0], rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("causal", [False, True])
def test_split_k_merge_associative(causal):
    """The split-K merge over any chunking and any merge order reproduces eq:kl-def."""
    d = inputs.make("tiny", n_q=64, n_k=150)
    w = d["w"]
    q1, k1, q2, k2 = (d[k][0, 0].astype(np.float64) for k in ("Q1", "K1", "Q2", "K2"))
    rk, r1, r2 = oracle.forward(d["Q1"], d["K1"], d["Q2"], d["K2"], w.s1, w.s2, causal, FWD)
    rng = np.random.default_rng(19)
    for W in (1, 2, 3, 5, 8):
        order = rng.permutation(W)
        kl, l1, l2 = oracle.split_merge_forward_head(q1, k1, q2, k2, w.s1, w.s2, causal, FWD, W, 16, order)
        np.testing.assert_allclose(kl, rk[0, 0], rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(l1, r1[0, 0], rtol=1e-13, atol=1e-13)
        np.testing.assert_allclose(l2, r2[0, 0], rtol=1e-13, atol=1e-13)


def test_acc_invariant_after_each_tile():
    """eq:acc-invariant: after tiles 1..j, acc = sum_{keys seen} e^{S1 - m1^(j)} (S1 - S2)."""
    from oracle import online_model as om
    d = inputs.make("tiny", n_q=16, n_k=64)
    w = d["w"]
    q1, k1, q2, k2 = (d[k][0, 0].astype(np.float64) for k in ("Q1", "K1", "Q2", "K2"))
    S1, S2 = om._logits(q1, k1, q2, k2, w.s1, w.s2)
    mask = np.ones_like(S1, dtype=bool)
    st = om.empty_state(16)
    for j0 in range(0, 64, 8):
        st = om.merge_states(st, om.tile_state(S1[:, j0:j0 + 8], S2[:, j0:j0 + 8], mask[:, j0:j0 + 8]))
        seen = slice(0, j0 + 8)
        m1 = S1[:, seen].max(axis=1)
        np.testing.assert_allclose(st["m1"], m1, rtol=0, atol=0)
        ref = (np.exp(S1[:, seen] - m1[:, None]) * (S1[:, seen] - S2[:, seen])).sum(axis=1)
        np.testing.assert_allclose(st["acc"], ref, rtol=1e-12, atol=1e-13)


def test_empty_partial_state_is_neutral():
    """A set of keys a row may not see gives the empty state, and merging it
    changes nothing: a causal row's tiles past its frontier, and a split-K
    chunk that holds none of its keys."""
    from oracle import online_model as om
    rng = np.random.default_rng(5)
    S1, S2 = rng.standard_normal((4, 6)), rng.standard_normal((4, 6))
    mask = np.ones((4, 6), dtype=bool)
    mask[1] = False           # row 1 sees none of these keys
    mask[2, 3:] = False
    t = om.tile_state(S1, S2, mask)
    assert np.isneginf(t["m1"][1]) and np.isneginf(t["m2"][1])
    assert t["l1"][1] == 0.0 and t["l2"][1] == 0.0 and t["acc"][1] == 0.0
    full = om.tile_state(S1, S2, np.ones((4, 6), dtype=bool))
    for a, b in ((om.merge_states(full, om.empty_state(4)), full), (om.merge_states(om.empty_state(4), full), full)):
        for k in full:
            np.testing.assert_array_equal(a[k], b[k])
    kl, l1, l2 = om.finalize(om.empty_state(3))
    assert np.all(kl == 0.0) and np.all(np.isneginf(l1)) and np.all(np.isneginf(l2))


def test_any_applied_exponent_reference_finalizes_the_same():
    """A partial state need not be relative to its maxima: with l_t = sum
    e^{S_t - u_t} and acc = sum e^{S1 - u1} (S1 - S2) over its keys, any
    applied references u_t merge (Sec. 3.3) and finalize (eq:kl-final) to
    the same KL and LSEs. The forward kernel relies on this: it reduces each
    tile against the reference its row already holds and forms new maxima
    only when a tile's terms would leave the fp32 range. Pinned against the
    plain definition, causal, with each tile either keeping the previous
    tile's reference (a merge with equal references is a plain addition, as
    in the kernel) or taking one up to 60 nats below or above its maximum."""
    from oracle import online_model as om
    from oracle.kl_oracle import allowed_mask
    n_q, n_k, bk = 24, 160, 32
    d = inputs.make("tiny", n_q=n_q, n_k=n_k)
    w = d["w"]
    q1, k1, q2, k2 = (d[k][0, 0].astype(np.float64) for k in ("Q1", "K1", "Q2", "K2"))
    rk, r1, r2 = oracle.forward(d["Q1"], d["K1"], d["Q2"], d["K2"], w.s1, w.s2, True, FWD)
    S1, S2 = om._logits(q1, k1, q2, k2, w.s1, w.s2)
    mask = allowed_mask(np.arange(n_q), n_q, n_k, True)
    rng = np.random.default_rng(23)
    st = om.empty_state(n_q)
    for j0 in range(0, n_k, bk):
        S1t, S2t, mt = S1[:, j0:j0 + bk], S2[:, j0:j0 + bk], mask[:, j0:j0 + bk]
        seen = mt.any(axis=1)
        refs = []
        for St, held in ((S1t, st["m1"]), (S2t, st["m2"])):
            fresh = np.where(mt, St, -np.inf).max(axis=1) + rng.uniform(-60.0, 60.0, n_q)
            keep = rng.random(n_q) < 0.6
            refs.append(np.where(seen, np.where(keep & np.isfinite(held), held, fresh), -np.inf))
        u1, u2 = refs
        e1 = np.where(mt, np.exp(np.where(mt, S1t, 0.0) - np.where(seen, u1, 0.0)[:, None]), 0.0)
        e2 = np.where(mt, np.exp(np.where(mt, S2t, 0.0) - np.where(seen, u2, 0.0)[:, None]), 0.0)
        tile = dict(m1=u1, l1=e1.sum(axis=1), m2=u2, l2=e2.sum(axis=1),
                    acc=(e1 * np.where(mt, S1t - S2t, 0.0)).sum(axis=1))
        st = om.merge_states(st, tile)
    kl, l1, l2 = om.finalize(st)
    np.testing.assert_allclose(kl, rk[0, 0], rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(l1, r1[0, 0], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(l2, r2[0, 0], rtol=1e-12, atol=1e-12)
