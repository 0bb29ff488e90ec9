"""Pins of the LM-head log-probability oracle and the objectives built on it
(oracle/lce_oracle.py), each against something other than the oracle itself:
torch's log_softmax / cross_entropy / autograd (independent implementations),
brute-force loops on tiny inputs, closed forms of the DiPO surrogate at its
special cases (ratio 1, clipped from either side, KL at the reference), the
invariants of a softmax gradient, and finite differences."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle


def _case(N, V, Dm, seed, scale=1.0):
    g = np.random.default_rng(seed)
    H = g.standard_normal((N, Dm)) * scale
    W = g.standard_normal((V, Dm)) / math.sqrt(Dm)
    t = g.integers(0, V, size=N)
    return H, W, t


def test_logprobs_match_torch_log_softmax():
    H, W, t = _case(7, 33, 16, 1)
    t[2], t[5] = -1, 33  # not scored
    logp, lse = oracle.lm_head_logprobs(H, W, t)
    logits = torch.from_numpy(H) @ torch.from_numpy(W).T
    ref = torch.log_softmax(logits, dim=1)
    np.testing.assert_allclose(lse, torch.logsumexp(logits, 1).numpy(), rtol=0, atol=1e-12)
    for n in range(7):
        want = 0.0 if t[n] in (-1, 33) else float(ref[n, t[n]])
        assert abs(logp[n] - want) < 1e-12


def test_lse_brute_force_tiny():
    H = np.array([[0.5, -1.0, 2.0], [0.0, 0.25, -0.5]])
    W = np.array([[1.0, 0.0, 0.0], [0.0, 1.0, 0.0], [0.0, 0.0, 1.0], [1.0, 1.0, 1.0], [-1.0, 0.5, 0.0]])
    t = np.array([3, 0])
    logp, lse = oracle.lm_head_logprobs(H, W, t)
    for n in range(2):
        z = [sum(H[n][d] * W[v][d] for d in range(3)) for v in range(5)]
        want = math.log(sum(math.exp(x) for x in z))
        assert abs(lse[n] - want) < 1e-13
        assert abs(logp[n] - (z[t[n]] - want)) < 1e-13


def test_logprobs_normalised_over_targets():
    H, W, _ = _case(3, 50, 8, 2)
    for n in range(3):
        lp = [oracle.lm_head_logprobs(H[n:n + 1], W, [v])[0][0] for v in range(50)]
        assert abs(sum(math.exp(x) for x in lp) - 1.0) < 1e-12


def test_large_logits_stay_finite():
    # logits of order 1e3: an unshifted exp would overflow
    H, W, t = _case(4, 20, 8, 3, scale=2000.0)
    logp, lse = oracle.lm_head_logprobs(H, W, t)
    logits = torch.from_numpy(H) @ torch.from_numpy(W).T
    assert np.all(np.isfinite(lse)) and np.all(np.isfinite(logp))
    ref = torch.log_softmax(logits, 1).numpy()
    np.testing.assert_allclose(logp, ref[np.arange(4), t], rtol=1e-12, atol=1e-9)


def test_backward_matches_torch_autograd():
    H, W, t = _case(6, 29, 12, 4)
    t[1] = -5
    c = np.random.default_rng(5).standard_normal(6)
    dH, dW = oracle.lm_head_backward(H, W, t, c)
    Ht = torch.from_numpy(H).requires_grad_()
    Wt = torch.from_numpy(W).requires_grad_()
    lp = torch.log_softmax(Ht @ Wt.T, 1)
    valid = torch.from_numpy((t >= 0) & (t < 29))
    tt = torch.from_numpy(np.where((t >= 0) & (t < 29), t, 0))
    picked = lp.gather(1, tt[:, None])[:, 0] * valid
    (picked * torch.from_numpy(c)).sum().backward()
    np.testing.assert_allclose(dH, Ht.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dW, Wt.grad.numpy(), rtol=1e-10, atol=1e-12)
    assert np.all(dH[1] == 0)  # a position that is not scored has no gradient


def test_backward_finite_differences():
    H, W, t = _case(3, 11, 5, 6)
    c = np.array([0.7, -1.3, 0.4])
    dH, dW = oracle.lm_head_backward(H, W, t, c)
    f = lambda H_, W_: float(np.dot(c, oracle.lm_head_logprobs(H_, W_, t)[0]))  # noqa: E731
    h = 1e-6
    for (i, j) in ((0, 0), (2, 4), (1, 2)):
        Hp, Hm = H.copy(), H.copy()
        Hp[i, j] += h
        Hm[i, j] -= h
        assert abs((f(Hp, W) - f(Hm, W)) / (2 * h) - dH[i, j]) < 1e-7
    for (i, j) in ((0, 0), (7, 3), (10, 1)):
        Wp, Wm = W.copy(), W.copy()
        Wp[i, j] += h
        Wm[i, j] -= h
        assert abs((f(H, Wp) - f(H, Wm)) / (2 * h) - dW[i, j]) < 1e-7


def test_backward_softmax_gradient_sums_to_zero_over_vocab():
    H, W, t = _case(5, 40, 9, 7)
    c = np.random.default_rng(8).standard_normal(5)
    _, dW = oracle.lm_head_backward(H, W, t, c)
    # each row of dlogits sums to zero, so the vocabulary rows of dW cancel
    assert np.abs(dW.sum(axis=0)).max() < 1e-12


def test_masked_ce_matches_torch_cross_entropy():
    H, W, t = _case(8, 31, 7, 9)
    w = np.random.default_rng(10).uniform(0, 2, 8) * (np.arange(8) % 3 != 0)  # w(t) times a mask
    logp, _ = oracle.lm_head_logprobs(H, W, t)
    loss, dl = oracle.masked_ce_objective(logp, w)
    logits = torch.from_numpy(H) @ torch.from_numpy(W).T
    ce = F.cross_entropy(logits, torch.from_numpy(t), reduction="none").numpy()
    np.testing.assert_allclose(loss, w * ce, rtol=1e-12, atol=1e-14)
    np.testing.assert_array_equal(dl, -w)


def test_dipo_online_update_ratio_one():
    # pi_old = sg(pi): r = 1, so s = A and the derivative of s is A (Eq. 7)
    g = np.random.default_rng(11)
    lp = -g.uniform(0.1, 5, 10)
    ref = lp + g.normal(0, 0.3, 10)
    A = g.normal(0, 1, 10)
    w = np.full(10, 0.1)
    beta = 0.04
    loss, dl = oracle.dipo_objective(lp, lp, ref, A, w, 0.2, beta)
    kl = np.exp(ref - lp) - (ref - lp) - 1
    np.testing.assert_allclose(loss, -w * (A - beta * kl), rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(dl, -w * (A - beta * (1 - np.exp(ref - lp))), rtol=1e-13, atol=1e-15)


def test_dipo_clipping_cases():
    eps = 0.2
    lp_old = np.zeros(4)
    # r = e^0.5 > 1 + eps with A > 0: clipped term (1 + eps) A is the minimum, no gradient
    # r = e^-0.5 < 1 - eps with A < 0: clipped term (1 - eps) A is the minimum, no gradient
    # r = e^0.5 with A < 0: the unclipped r A is the minimum
    # r = e^0.1 inside the range: both terms agree, gradient r A
    lp = np.array([0.5, -0.5, 0.5, 0.1])
    A = np.array([1.0, -1.0, -1.0, 2.0])
    w = np.ones(4)
    loss, dl = oracle.dipo_objective(lp, lp_old, None, A, w, eps, 0.0)
    r = np.exp(lp)
    np.testing.assert_allclose(loss, [-(1 + eps), (1 - eps), r[2], -r[3] * 2.0], rtol=1e-13)
    np.testing.assert_allclose(dl, [0.0, 0.0, r[2], -2.0 * r[3]], rtol=1e-13, atol=0)


def test_dipo_kl_estimator_properties_and_finite_differences():
    g = np.random.default_rng(12)
    lp = -g.uniform(0.1, 3, 50)
    ref = lp + g.normal(0, 1, 50)
    A = g.normal(0, 1, 50)
    w = g.uniform(0.5, 1.5, 50)
    old = lp + g.normal(0, 0.05, 50)  # ratios near 1, away from the clip edges
    beta = 0.3
    # KL is zero at the reference and non-negative elsewhere
    z, _ = oracle.dipo_objective(lp, lp, lp, np.zeros(50), w, 0.2, 1.0)
    assert np.abs(z).max() < 1e-15
    kl_only, _ = oracle.dipo_objective(lp, lp, ref, np.zeros(50), np.ones(50), 0.2, 1.0)
    assert np.all(kl_only >= 0)
    loss, dl = oracle.dipo_objective(lp, old, ref, A, w, 0.2, beta)
    h = 1e-6
    lp_p, _ = oracle.dipo_objective(lp + h, old, ref, A, w, 0.2, beta)
    lp_m, _ = oracle.dipo_objective(lp - h, old, ref, A, w, 0.2, beta)
    r = np.exp(lp - old)
    away = np.abs(r - 0.8) > 1e-3
    away &= np.abs(r - 1.2) > 1e-3
    np.testing.assert_allclose(((lp_p - lp_m) / (2 * h))[away], dl[away], rtol=1e-6, atol=1e-8)


def test_sampled_matches_full_evaluation():
    H, W, t = _case(9, 70, 6, 13)
    t[4] = -1
    rows = [1, 4, 7]
    c = np.zeros(9)
    c[rows] = [0.5, 2.0, -1.5]
    logp, lse = oracle.lm_head_logprobs(H, W, t)
    dH, dW = oracle.lm_head_backward(H, W, t, c)
    vr = [0, 5, 33, 69]
    slp, slse, sdH, sdW = oracle.lm_head_sampled(H, W, t, c, rows, vr, chunk=16)
    np.testing.assert_allclose(slp, logp[rows], rtol=0, atol=1e-12)
    np.testing.assert_allclose(slse, lse[rows], rtol=0, atol=1e-12)
    np.testing.assert_allclose(sdH, dH[rows], rtol=0, atol=1e-12)
    np.testing.assert_allclose(sdW, dW[vr], rtol=0, atol=1e-12)
