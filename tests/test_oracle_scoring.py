"""Pins of the oracle's logits, log-softmax statistics and two-policy scoring.

References that do not share the oracle's code: numpy matmul of decoded
operands (torch's float8 decoding for mu), scipy's logsumexp / entropy,
math.fsum brute force for V <= 16, and closed forms (uniform logits, a
lossless mu that must reproduce pi exactly, Sec. 3.1: E = 0 iff the two
policies give identical probabilities).
"""
import math

import numpy as np
import pytest
import scipy.special
import scipy.stats

import inputs
import oracle


def _bf16(x):
    return inputs.float_to_bf16_bits(np.asarray(x, np.float32))


def _dec_fp8(q):
    import torch
    return torch.from_numpy(np.ascontiguousarray(q)).view(torch.float8_e4m3fn).to(torch.float64).numpy()


def test_logits_pi_matches_numpy_matmul_nonsquare():
    r = np.random.default_rng(1)
    V, d = 37, 24
    h = _bf16(r.standard_normal(d))
    w = _bf16(r.standard_normal((V, d)) * 0.3)
    z = oracle.logits_pi(h, w, inv_temperature=1.0 / 0.7)
    want = (oracle.bf16_to_float(w).astype(np.float64) @ oracle.bf16_to_float(h).astype(np.float64)) / 0.7
    np.testing.assert_allclose(z, want, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("scaling", [oracle.PER_TENSOR, oracle.PER_ROW, oracle.MX32])
def test_logits_mu_matches_torch_decoded_matmul(scaling):
    pytest.importorskip("torch")
    r = np.random.default_rng(2)
    T, V, d = 3, 29, 64
    h = _bf16(r.standard_normal((T, d)) * 2)
    w = _bf16(r.standard_normal((V, d)) * 0.2)
    hq, hs = oracle.quantize_fp8(h, scaling)
    wq, ws = oracle.quantize_fp8(w, scaling)
    a = _dec_fp8(hq)
    b = _dec_fp8(wq)
    if scaling == oracle.PER_TENSOR:
        a, b = a * float(hs[0]), b * float(ws[0])
    elif scaling == oracle.PER_ROW:
        a, b = a * hs.astype(np.float64)[:, None], b * ws.astype(np.float64)[:, None]
    else:
        a = a * np.repeat(np.ldexp(1.0, hs.astype(np.int64) - 127), 32, axis=1)
        b = b * np.repeat(np.ldexp(1.0, ws.astype(np.int64) - 127), 32, axis=1)
    want = a @ b.T * 1.25
    for t in range(T):
        rs = oracle._row_scale(hs, scaling, t)
        z = oracle.logits_mu(hq[t], rs, wq, ws, scaling, inv_temperature=1.25)
        np.testing.assert_allclose(z, want[t], rtol=1e-12, atol=1e-12)


def test_token_stats_match_scipy():
    r = np.random.default_rng(3)
    for V in (1, 2, 5, 16, 1000):
        z = r.standard_normal(V) * 4
        for tid in {0, V // 2, V - 1}:
            lse, lp, H = oracle.token_stats(z, tid)
            assert abs(lse - scipy.special.logsumexp(z)) < 1e-12 * max(1, abs(lse))
            p = scipy.special.softmax(z)
            assert abs(lp - math.log(p[tid])) < 1e-11
            assert abs(H - scipy.stats.entropy(p)) < 1e-11


def test_token_stats_brute_force_small_vocab():
    r = np.random.default_rng(4)
    for V in range(1, 17):
        z = r.uniform(-20, 20, V)
        tid = int(r.integers(V))
        e = [math.exp(v) for v in z]
        S = math.fsum(e)
        p = [v / S for v in e]
        lse, lp, H = oracle.token_stats(z, tid)
        assert abs(sum(p) - 1) < 1e-12
        assert abs(lse - math.log(S)) < 1e-12
        assert abs(lp - math.log(p[tid])) < 1e-12
        assert abs(H - math.fsum(-q * math.log(q) for q in p if q > 0)) < 1e-12
        assert -1e-15 <= H <= math.log(V) + 1e-12


def test_uniform_logits_closed_form():
    for V in (1, 7, 2048, 151936):
        lse, lp, H = oracle.token_stats(np.full(V, 0.0), V - 1)
        assert abs(lp + math.log(V)) < 1e-9 and abs(H - math.log(V)) < 1e-9


def test_dominant_logit_gives_zero_entropy():
    z = np.zeros(100)
    z[42] = 1e3
    lse, lp, H = oracle.token_stats(z, 42)
    assert abs(lp) < 1e-12 and abs(H) < 1e-12


def test_shift_invariance():
    z = np.random.default_rng(5).standard_normal(300)
    a = oracle.token_stats(z, 11)
    b = oracle.token_stats(z + 123.25, 11)
    assert abs(a[1] - b[1]) < 1e-11 and abs(a[2] - b[2]) < 1e-10


def _lossless_case(T, V, d, seed):
    """H and W whose entries are e4m3 values and whose per-row (and overall)
    maximum is 448, so every FP8 scale is 1 and quantization is exact."""
    r = np.random.default_rng(seed)
    vals = oracle.e4m3_decode(np.arange(0x7F, dtype=np.uint8))
    small = vals[(vals <= 2.0)]
    h = r.choice(np.concatenate([small, -small]), size=(T, d)).astype(np.float32)
    w = r.choice(np.concatenate([small, -small]), size=(V, d)).astype(np.float32) / 64
    h[:, 0] = 448.0
    w[:, 0] = 448.0 / 64  # exact in bf16; rescaled to 448 by the per-row scale
    return _bf16(h), _bf16(w)


def test_lossless_mu_equals_pi():
    # mu computed from exactly-representable operands must equal pi:
    # log-ratio == 0 and d == 0 (Sec. 3.1: E = 0 <=> identical probabilities).
    T, V, d = 6, 50, 32
    h, w = _lossless_case(T, V, d, 6)
    ids = np.arange(T, dtype=np.int32) * 7 % V
    for scaling in (oracle.PER_ROW, oracle.MX32):
        hq, hs = oracle.quantize_fp8(h, scaling)
        wq, ws = oracle.quantize_fp8(w, scaling)
        out = oracle.score(h, w, hq, hs, wq, ws, scaling, ids)
        np.testing.assert_array_equal(out["logp_pi"], out["logp_mu"])
        np.testing.assert_array_equal(out["ent_pi"], out["ent_mu"])


def test_score_composes_logits_and_stats_with_mask():
    w_ = inputs.WORKLOADS["tiny"]
    T = 10
    h = inputs.hidden_bf16(w_, T)
    w = inputs.weights_bf16(w_)
    ids = inputs.uniform_ids(w_, T)
    msk = np.array([1, 1, 0, 1, 1, 1, 1, 0, 1, 1], np.uint8)
    hq, hs = oracle.quantize_fp8(h, oracle.PER_ROW)
    wq, ws = oracle.quantize_fp8(w, oracle.PER_ROW)
    out = oracle.score(h, w, hq, hs, wq, ws, oracle.PER_ROW, ids, msk)
    # reference: numpy float64 logits + scipy statistics
    Hf = oracle.bf16_to_float(h).astype(np.float64)
    Wf = oracle.bf16_to_float(w).astype(np.float64)
    zp = Hf @ Wf.T
    zm = (_dec_fp8(hq) * hs.astype(np.float64)[:, None]) @ (_dec_fp8(wq) * ws.astype(np.float64)[:, None]).T
    for t in range(T):
        if not msk[t]:
            assert out["logp_pi"][t] == 0 and out["ent_mu"][t] == 0
            continue
        for z, tag in ((zp[t], "pi"), (zm[t], "mu")):
            lse = scipy.special.logsumexp(z)
            assert abs(out["lse_" + tag][t] - lse) < 1e-10
            assert abs(out["logp_" + tag][t] - (z[ids[t]] - lse)) < 1e-10
            assert abs(out["ent_" + tag][t] - scipy.stats.entropy(scipy.special.softmax(z))) < 1e-9
            assert abs(out["z_" + tag][t] - z[ids[t]]) < 1e-10


def test_exact_integer_logits():
    # small integers are exact in bf16 and e4m3; logits are exact integers
    r = np.random.default_rng(7)
    T, V, d = 4, 40, 64
    h = r.integers(-4, 5, size=(T, d)).astype(np.float32)
    w = r.integers(-4, 5, size=(V, d)).astype(np.float32)
    z = oracle.logits_pi(_bf16(h[1]), _bf16(w))
    assert np.array_equal(z, (w.astype(np.int64) @ h[1].astype(np.int64)).astype(np.float64))


def test_sampler_picks_by_cumulative_probability():
    z = np.log(np.array([[0.1, 0.2, 0.3, 0.4]]))
    for u, want in ((0.0, 0), (0.05, 0), (0.1000001, 1), (0.35, 2), (0.61, 3), (0.999, 3)):
        assert oracle.sample_inverse_cdf(z, np.array([u]))[0] == want
