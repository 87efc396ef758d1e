"""Pins of the oracle's ACRL-weighted surrogate (Eq. ACRL, Sec. 4.1) and of
its LM-head backward, checked against what the mathematics fixes: closed
forms of the clipped objective, the batch aggregation of means, central
finite differences of the oracle's own loss, PyTorch's fp64 autograd of the
log-softmax (a library routine), and invariants of the softmax gradient."""
import math

import numpy as np
import pytest

import oracle
from cases import random_bf16

EPS = 0.2


def _one_token_case(A, r, eps_low=EPS, eps_high=EPS, w=1.0):
    """One prompt, one response of one token: c_t = 1."""
    lp_old = np.array([-1.0])
    lp_new = lp_old + math.log(r)
    coef, loss = oracle.surrogate(1, 1, np.ones(1), np.zeros(1), 1, lp_new, lp_old, np.array([A]),
                                  weight=np.array([w]), eps_low=eps_low, eps_high=eps_high)
    return coef[0], loss


@pytest.mark.parametrize("A,r,term,grad", [
    # A > 0: min(r, clip(r)) A -- the ratio is capped above at 1 + eps
    (1.0, 1.5, 1.2, 0.0),     # clipped above: constant 1.2 A, no gradient
    (1.0, 0.5, 0.5, 0.5),     # r < 1 - eps: the unclipped r A is the smaller
    (1.0, 1.1, 1.1, 1.1),     # inside the range: both terms equal, r A
    # A < 0: max(r, clip(r)) A -- the ratio is capped below at 1 - eps
    (-1.0, 1.5, -1.5, -1.5),  # r > 1 + eps: r A is the smaller, gradient r A
    (-1.0, 0.5, -0.8, 0.0),   # clipped below: constant 0.8 A
    (0.0, 1.3, 0.0, 0.0),     # no advantage, no gradient
])
def test_clip_cases(A, r, term, grad):
    coef, loss = _one_token_case(A, r)
    # loss = -J; coef = d loss / d logp_new = -(d term / d logp_new)
    assert loss == pytest.approx(-term, abs=1e-12)
    assert coef == pytest.approx(-grad, abs=1e-12)


def test_asymmetric_clip_range():
    # a clip-higher range (eps_high > eps_low) keeps r = 1.25 unclipped for A > 0
    coef, loss = _one_token_case(1.0, 1.25, eps_low=0.2, eps_high=0.28)
    assert loss == pytest.approx(-1.25) and coef == pytest.approx(-1.25)
    coef, loss = _one_token_case(1.0, 1.25, eps_low=0.2, eps_high=0.2)
    assert loss == pytest.approx(-1.2) and coef == 0.0
    coef, loss = _one_token_case(-1.0, 0.75, eps_low=0.2, eps_high=0.28)
    assert loss == pytest.approx(0.8) and coef == 0.0


def test_weight_scales_term_and_gradient():
    c1, l1 = _one_token_case(1.0, 0.9)
    c3, l3 = _one_token_case(1.0, 0.9, w=3.0)
    assert l3 == pytest.approx(3 * l1) and c3 == pytest.approx(3 * c1)


def _batch(lengths, groups, L):
    B = len(lengths)
    m = np.zeros((B, L), np.uint8)
    for i, n in enumerate(lengths):
        m[i, :n] = 1
    return m, np.asarray(groups, np.int32)


def test_mean_of_means_is_one_for_unit_terms():
    # A = 1, r = 1, w = 1: every term is 1 and J is a mean of means of means
    m, g = _batch([3, 0, 7, 1, 5, 2], [0, 0, 1, 1, 3, 3], 8)  # group 2 and a response empty
    B, L = m.shape
    lp = np.random.default_rng(0).standard_normal(B * L)
    coef, loss = oracle.surrogate(B, L, m, g, 4, lp, lp, np.ones(B))
    assert loss == pytest.approx(-1.0, abs=1e-14)
    assert coef.sum() == pytest.approx(-1.0, abs=1e-14)
    assert np.all(coef[m.ravel() == 0] == 0)


def test_group_means_weight_prompts_equally():
    # r = 1: the term of a token is A, so J = mean over prompts of the
    # prompt's mean of A over its responses, whatever their lengths
    m, g = _batch([2, 4, 3], [0, 0, 1], 4)
    B, L = m.shape
    lp = np.zeros(B * L)
    adv = np.array([1.0, 3.0, 2.0])
    coef, loss = oracle.surrogate(B, L, m, g, 2, lp, lp, adv)
    assert loss == pytest.approx(-((1.0 + 3.0) / 2 + 2.0) / 2)
    # per token: -A / (n_prompts G |a_i|)
    np.testing.assert_allclose(coef.reshape(B, L)[0, :2], -1.0 / (2 * 2 * 2))
    np.testing.assert_allclose(coef.reshape(B, L)[1, :4], -3.0 / (2 * 2 * 4))
    np.testing.assert_allclose(coef.reshape(B, L)[2, :3], -2.0 / (2 * 1 * 3))


def test_coefficient_is_the_derivative_of_the_loss():
    rng = np.random.default_rng(5)
    m, g = _batch([5, 3, 6, 2], [0, 0, 1, 1], 6)
    B, L = m.shape
    lp_old = rng.normal(-2.0, 0.5, B * L)
    lp_new = lp_old + rng.normal(0.0, 0.3, B * L)
    adv = rng.standard_normal(B * L)
    wt = rng.uniform(0.5, 3.0, B * L)
    args = dict(adv_per_token=True, weight=wt, eps_low=0.2, eps_high=0.28)
    coef, _ = oracle.surrogate(B, L, m, g, 2, lp_new, lp_old, adv, **args)
    h = 1e-6
    checked = 0
    for t in np.flatnonzero(m.ravel()):
        r = math.exp(lp_new[t] - lp_old[t])
        if min(abs(r - 0.8), abs(r - 1.28)) < 1e-3:
            continue  # a kink of the clipped term
        up, dn = lp_new.copy(), lp_new.copy()
        up[t] += h
        dn[t] -= h
        lu = oracle.surrogate(B, L, m, g, 2, up, lp_old, adv, **args)[1]
        ld = oracle.surrogate(B, L, m, g, 2, dn, lp_old, adv, **args)[1]
        assert coef[t] == pytest.approx((lu - ld) / (2 * h), rel=1e-6, abs=1e-9)
        checked += 1
    assert checked >= 12
    # both branches occur in this case
    assert np.any(coef[m.ravel() == 1] == 0) and np.any(coef[m.ravel() == 1] != 0)


def test_surrogate_rejects_bad_arguments():
    m, g = _batch([2], [0], 2)
    lp = np.zeros(2)
    with pytest.raises(ValueError):
        oracle.surrogate(1, 2, m, np.array([3]), 1, lp, lp, np.ones(1))
    with pytest.raises(ValueError):
        oracle.surrogate(1, 2, m, g, 1, lp, lp, np.ones(1), eps_low=-0.1)


# ------------------------------------------------------------ LM-head backward
def _backward_case(n, d, V, seed, inv_temperature=1.0):
    H = random_bf16((n, d), seed)
    W = random_bf16((V, d), seed + 1, std=2.5 / math.sqrt(d))
    rng = np.random.default_rng(seed + 2)
    ids = rng.integers(0, V, n).astype(np.int32)
    coef = rng.standard_normal(n)
    return H, W, ids, coef


def test_backward_matches_torch_autograd():
    torch = pytest.importorskip("torch")
    n, d, V, itau = 7, 24, 37, 1.0 / 0.7
    H, W, ids, coef = _backward_case(n, d, V, 11, itau)
    dh, dw = oracle.lm_head_backward(H, W, ids, coef, itau)
    h = torch.tensor(oracle.bf16_to_float(H), dtype=torch.float64, requires_grad=True)
    w = torch.tensor(oracle.bf16_to_float(W), dtype=torch.float64, requires_grad=True)
    lp = torch.log_softmax(h @ w.T * itau, dim=1)[torch.arange(n), torch.from_numpy(ids).long()]
    phi = (torch.from_numpy(coef) * lp).sum()
    phi.backward()
    np.testing.assert_allclose(dh, h.grad.numpy(), rtol=1e-10, atol=1e-14)
    np.testing.assert_allclose(dw, w.grad.numpy(), rtol=1e-10, atol=1e-14)


def test_backward_two_word_vocabulary_closed_form():
    # V = 2: log p_a = -log(1 + exp(z_b - z_a)), so
    # d/dh = coef (1 - p_a) (W_a - W_b) / tau
    d, itau = 16, 2.0
    H, W, ids, coef = _backward_case(1, d, 2, 3)
    ids[:] = 1
    h = oracle.bf16_to_float(H)[0].astype(np.float64)
    w = oracle.bf16_to_float(W).astype(np.float64)
    z = w @ h * itau
    pa = 1.0 / (1.0 + math.exp(z[0] - z[1]))
    dh, dw = oracle.lm_head_backward(H, W, ids, coef, itau)
    np.testing.assert_allclose(dh[0], coef[0] * (1 - pa) * (w[1] - w[0]) * itau, rtol=1e-12)
    np.testing.assert_allclose(dw[1], coef[0] * (1 - pa) * h * itau, rtol=1e-12)
    np.testing.assert_allclose(dw[0], -coef[0] * (1 - pa) * h * itau, rtol=1e-12)


def test_backward_invariants():
    n, d, V = 9, 32, 53
    H, W, ids, coef = _backward_case(n, d, V, 21)
    dh, dw, dha, dwa = oracle.lm_head_backward(H, W, ids, coef, 1.0, want_abs=True)
    # every row of dZ sums to zero, so the vocabulary rows of dW do too
    np.testing.assert_allclose(dw.sum(axis=0), 0.0, atol=1e-12)
    assert np.all(np.abs(dh) <= dha * (1 + 1e-12)) and np.all(np.abs(dw) <= dwa * (1 + 1e-12))
    # identical vocabulary rows: a uniform softmax and no gradient reaching H
    W1 = np.repeat(W[:1], V, axis=0)
    dh1, _ = oracle.lm_head_backward(H, W1, ids, coef, 1.0)
    np.testing.assert_allclose(dh1, 0.0, atol=1e-13)
    # no coefficient, no gradient
    dh0, dw0 = oracle.lm_head_backward(H, W, ids, np.zeros(n), 1.0)
    assert not dh0.any() and not dw0.any()
    # rows chosen one by one agree with the full result
    dhs, dws = oracle.lm_head_backward(H, W, ids, coef, 1.0, hrows=[4, 0], wrows=[52, 7])
    np.testing.assert_array_equal(dhs, dh[[4, 0]])
    np.testing.assert_array_equal(dws, dw[[52, 7]])


def test_backward_rejects_out_of_range_ids():
    H, W, ids, coef = _backward_case(2, 8, 5, 1)
    ids[1] = 5
    with pytest.raises(ValueError):
        oracle.lm_head_backward(H, W, ids, coef)
