"""Pins of the oracle's full-vocabulary discrepancy measures (KL in both
directions and the Euclidean distance between softmax(z_pi) and
softmax(z_mu); the measures the paper names beside its absolute distance).
Checked against a closed form, SciPy's relative entropy and Euclidean
distance (library routines), Pinsker's inequality, the second-order
expansion of KL, and the special cases that must give zero."""
import math

import numpy as np
import pytest
from scipy.spatial.distance import euclidean
from scipy.special import rel_entr, softmax

import inputs
import oracle
from cases import lossless_integer_case, random_bf16


def _sig(x):
    return 1.0 / (1.0 + math.exp(-x))


@pytest.mark.parametrize("x,y", [(1.0, 1.2), (-3.0, 2.5), (0.0, 0.0), (7.0, -7.0)])
def test_two_word_closed_form(x, y):
    # logits (0, x) and (0, y): Bernoulli(a) and Bernoulli(b), a = sigmoid(x)
    a, b = _sig(x), _sig(y)
    kl_ab = a * math.log(a / b) + (1 - a) * math.log((1 - a) / (1 - b))
    kl_ba = b * math.log(b / a) + (1 - b) * math.log((1 - b) / (1 - a))
    k1, k2, l2 = oracle.token_divergence([0.0, x], [0.0, y])
    assert k1 == pytest.approx(kl_ab, rel=1e-12, abs=1e-15)
    assert k2 == pytest.approx(kl_ba, rel=1e-12, abs=1e-15)
    assert l2 == pytest.approx(math.sqrt(2.0) * abs(a - b), rel=1e-12, abs=1e-15)


@pytest.mark.parametrize("V,scale", [(5, 1.0), (16, 3.0), (1000, 2.5), (30000, 2.5)])
def test_matches_scipy(V, scale):
    r = np.random.default_rng(V)
    zp = r.normal(0, scale, V)
    zm = zp + r.normal(0, 0.3, V)
    p, q = softmax(zp), softmax(zm)
    k1, k2, l2 = oracle.token_divergence(zp, zm)
    assert k1 == pytest.approx(rel_entr(p, q).sum(), rel=1e-9)
    assert k2 == pytest.approx(rel_entr(q, p).sum(), rel=1e-9)
    assert l2 == pytest.approx(euclidean(p, q), rel=1e-9)


def test_invariants():
    r = np.random.default_rng(3)
    zp = r.normal(0, 2.5, 2048)
    zm = zp + r.normal(0, 0.2, 2048)
    k1, k2, l2 = oracle.token_divergence(zp, zm)
    assert k1 > 0 and k2 > 0 and l2 > 0
    # shifting a policy's logits changes nothing
    s1 = oracle.token_divergence(zp + 17.0, zm - 4.0)
    np.testing.assert_allclose(s1, (k1, k2, l2), rtol=1e-9)
    # swapping the policies swaps the two directions
    s2 = oracle.token_divergence(zm, zp)
    np.testing.assert_allclose(s2, (k2, k1, l2), rtol=1e-12)
    # Pinsker: L2 <= L1 <= sqrt(2 KL), both directions
    l1 = np.abs(softmax(zp) - softmax(zm)).sum()
    assert l2 <= l1 <= math.sqrt(2 * k1) and l1 <= math.sqrt(2 * k2)
    # identical policies
    assert oracle.token_divergence(zp, zp) == (0.0, 0.0, 0.0)


def test_second_order_expansion():
    # KL(pi || mu) = Var_pi(z_mu - z_pi) / 2 + O(eps^3) for logits eps apart
    r = np.random.default_rng(4)
    zp = r.normal(0, 2.5, 4096)
    delta = r.normal(0, 1.0, 4096)
    p = softmax(zp)
    var = p @ delta ** 2 - (p @ delta) ** 2
    for eps in (1e-2, 1e-3):
        k1, k2, _ = oracle.token_divergence(zp, zp + eps * delta)
        assert k1 == pytest.approx(0.5 * eps * eps * var, rel=5 * eps)
        assert k2 == pytest.approx(0.5 * eps * eps * var, rel=5 * eps)


def test_rows_driver_and_lossless_operands():
    # the rows driver gives the per-token values of the logits' divergences
    w = inputs.WORKLOADS["tiny"]
    H = random_bf16((7, w.d), 5)
    W = random_bf16((300, w.d), 6, std=2.5 / math.sqrt(w.d))
    hq, hs = oracle.quantize_fp8(H, oracle.PER_ROW)
    wq, ws = oracle.quantize_fp8(W, oracle.PER_ROW)
    mask = np.array([1, 1, 0, 1, 1, 1, 0], np.uint8)
    out = oracle.divergence(H, W, hq, hs, wq, ws, oracle.PER_ROW, mask=mask, inv_temperature=1.0 / 0.7)
    for r in range(7):
        if not mask[r]:
            assert out["kl_pi_mu"][r] == 0 and out["kl_mu_pi"][r] == 0 and out["l2"][r] == 0
            continue
        zp = oracle.logits_pi(H[r], W, 1.0 / 0.7)
        zm = oracle.logits_mu(hq[r], oracle._row_scale(hs, oracle.PER_ROW, r), wq, ws, oracle.PER_ROW, 1.0 / 0.7)
        np.testing.assert_allclose((out["kl_pi_mu"][r], out["kl_mu_pi"][r], out["l2"][r]),
                                   oracle.token_divergence(zp, zm), rtol=1e-12)
        assert out["kl_pi_mu"][r] > 0
    # operands exact in both formats: mu = pi and every measure is 0 (Sec. 3.1:
    # E = 0 exactly when the probabilities are identical)
    h, wb, _ = lossless_integer_case(5, 64, 32, 7)
    for sc in (oracle.PER_TENSOR, oracle.PER_ROW):
        hq, hs = oracle.quantize_fp8(h, sc)
        wq, ws = oracle.quantize_fp8(wb, sc)
        out = oracle.divergence(h, wb, hq, hs, wq, ws, sc, inv_temperature=1e-3)
        for k in out:
            assert np.all(out[k] == 0), k
