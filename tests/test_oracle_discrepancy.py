"""Pins of the oracle's discrepancy reduce and ACRL controller (no GPU).

Reduce: checked against a brute force over Python lists (per sequence,
group and batch, straight from Sec. 4.1's formulas for d, Y and X), numpy's
population std, and invariants (sum of lengths, equal-length groups).
Controller: the paper's own quadrant sign tables (Sec. 4.2, stored under
tests/golden/), hand-computed worked values, the clip at C, and identities
(alpha == 0 cases give weight 1; gamma = 1, Y = 0, A > 0 gives TIS).
"""
import math
import os

import numpy as np
import pytest

import inputs
import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _random_batch(B, L, n_groups, seed, empty_seq=None):
    r = np.random.default_rng(seed)
    lens = r.integers(1, L + 1, size=B)
    if empty_seq is not None:
        lens[empty_seq] = 0
    mask = (np.arange(L)[None, :] < lens[:, None]).astype(np.uint8)
    lp_pi = np.log(r.uniform(1e-4, 1, size=(B, L)))
    lp_mu = lp_pi + r.normal(0, 0.05, size=(B, L))
    lp_mu = np.minimum(lp_mu, 0.0)
    ent_pi = r.uniform(0, 5, size=(B, L))
    ent_mu = r.uniform(0, 5, size=(B, L))
    g = np.sort(r.integers(0, n_groups, size=B)).astype(np.int32)
    return mask, lp_pi, lp_mu, ent_pi, ent_mu, g


def _brute(B, L, mask, lp_pi, lp_mu, ent_pi, ent_mu, g, n_groups):
    seq = []
    toks = []
    for i in range(B):
        ds = [abs(math.exp(lp_pi[i, j]) - math.exp(lp_mu[i, j])) for j in range(L) if mask[i, j]]
        lr = [lp_pi[i, j] - lp_mu[i, j] for j in range(L) if mask[i, j]]
        toks += [(abs(math.exp(lp_pi[i, j]) - math.exp(lp_mu[i, j])), ent_pi[i, j], ent_mu[i, j],
                  lp_pi[i, j] - lp_mu[i, j]) for j in range(L) if mask[i, j]]
        seq.append((len(ds), math.fsum(ds), math.fsum(lr), math.fsum(ds) / len(ds) if ds else 0.0))
    gy = []
    for k in range(n_groups):
        members = [seq[i][3] for i in range(B) if g[i] == k and seq[i][0] > 0]
        gy.append((math.fsum(members) / len(members)) if members else None)
    ne = [y for y in gy if y is not None]
    return seq, gy, (math.fsum(ne) / len(ne) if ne else 0.0), toks


@pytest.mark.parametrize("seed,empty", [(1, None), (2, 3), (3, 0)])
def test_reduce_matches_brute_force(seed, empty):
    B, L, ng = 9, 23, 4
    mask, lp_pi, lp_mu, ent_pi, ent_mu, g = _random_batch(B, L, ng, seed, empty)
    out = oracle.discrepancy_reduce(B, L, lp_pi, lp_mu, mask, g, ng, ent_pi, ent_mu)
    seq, gy, yb, toks = _brute(B, L, mask, lp_pi, lp_mu, ent_pi, ent_mu, g, ng)
    for i in range(B):
        assert out["seq_len"][i] == seq[i][0]
        assert abs(out["seq_sum_d"][i] - seq[i][1]) < 1e-12
        assert abs(out["seq_sum_logratio"][i] - seq[i][2]) < 1e-12
        assert abs(out["seq_mean_d"][i] - seq[i][3]) < 1e-12
    for k in range(ng):
        if gy[k] is None:
            assert out["group_nseq"][k] == 0 and out["group_y"][k] == 0
        else:
            assert abs(out["group_y"][k] - gy[k]) < 1e-12
    st = out["stats"]
    d = np.array([t[0] for t in toks])
    assert abs(st[oracle.STAT_Y_BATCH] - yb) < 1e-12
    assert abs(st[oracle.STAT_TOK_MEAN_D] - d.mean()) < 1e-12
    assert st[oracle.STAT_TOK_MAX_D] == d.max()
    assert abs(st[oracle.STAT_TOK_STD_D] - np.std(d, ddof=0)) < 1e-12
    assert abs(st[oracle.STAT_MEAN_H_PI] - np.mean([t[1] for t in toks])) < 1e-12
    assert abs(st[oracle.STAT_MEAN_H_MU] - np.mean([t[2] for t in toks])) < 1e-12
    assert abs(st[oracle.STAT_TOK_MEAN_LOGRATIO] - np.mean([t[3] for t in toks])) < 1e-12
    assert st[oracle.STAT_N_TOKENS] == mask.sum()
    assert st[oracle.STAT_N_SEQS] == sum(1 for s in seq if s[0] > 0)
    assert st[oracle.STAT_N_GROUPS] == sum(1 for y in gy if y is not None)
    assert out["seq_len"].sum() == mask.sum()
    assert np.all(out["d_tok"].reshape(B, L)[mask == 0] == 0)


def test_equal_lengths_group_mean_is_token_mean():
    B, L, G = 8, 16, 4
    r = np.random.default_rng(4)
    mask = np.ones((B, L), np.uint8)
    mask[:, 12:] = 0
    lp_pi = np.log(r.uniform(0.01, 1, (B, L)))
    lp_mu = np.log(r.uniform(0.01, 1, (B, L)))
    g = (np.arange(B) // G).astype(np.int32)
    out = oracle.discrepancy_reduce(B, L, lp_pi, lp_mu, mask, g, 2)
    d = out["d_tok"].reshape(B, L)
    for k in range(2):
        assert abs(out["group_y"][k] - d[k * G:(k + 1) * G, :12].mean()) < 1e-13


def test_identical_policies_give_zero_discrepancy():
    B, L = 3, 10
    mask, lp, _, _, _, g = _random_batch(B, L, 2, 5)
    out = oracle.discrepancy_reduce(B, L, lp, lp, mask, g, 2)
    assert np.all(out["d_tok"] == 0) and np.all(out["seq_sum_logratio"] == 0)
    assert out["stats"][oracle.STAT_Y_BATCH] == 0


def test_distance_bounded_by_one():
    B, L = 4, 50
    mask, lp_pi, lp_mu, _, _, g = _random_batch(B, L, 1, 6)
    out = oracle.discrepancy_reduce(B, L, lp_pi, np.log(np.random.default_rng(0).uniform(1e-9, 1, (B, L))),
                                    mask, g, 1)
    assert np.all((out["d_tok"] >= 0) & (out["d_tok"] <= 1))


def test_reference_x_is_mean_of_nonempty_groups():
    gy = np.array([0.01, 0.0, 0.02, 0.03])
    gn = np.array([8, 0, 8, 8], np.int32)
    assert abs(oracle.reference_x(gy, gn) - 0.02) < 1e-15


def test_reference_x_equals_batch_y_of_step0():
    w = inputs.WORKLOADS["tiny"]
    B, L = 8, 20
    mask, lp_pi, lp_mu, _, _, g = _random_batch(B, L, 3, 7)
    out = oracle.discrepancy_reduce(B, L, lp_pi, lp_mu, mask, g, 3)
    X = oracle.reference_x(out["group_y"], out["group_nseq"])
    assert abs(X - out["stats"][oracle.STAT_Y_BATCH]) < 1e-15
    del w


# ------------------------------------------------------------------ controller
def _ctrl_one(pi, mu, A, Y, X, gamma, C):
    alpha, w = oracle.controller_step(1, 1, np.ones(1, np.uint8), np.zeros(1, np.int32),
                                      np.log([pi]), np.log([mu]), np.array([A]), False,
                                      oracle.Y_BATCH, None, None,
                                      np.array([Y] + [0.0] * (oracle.N_STATS - 1)), X, gamma, C)
    return alpha[0], w[0]


def _quadrant_rows():
    rows = []
    with open(os.path.join(GOLDEN, "acrl_quadrants.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                rows.append(line.split())
    assert len(rows) == 8
    return rows


@pytest.mark.parametrize("row", _quadrant_rows(), ids=lambda r: "%s-%s" % (r[0], r[1]))
def test_quadrant_signs_from_the_paper(row):
    regime, _, sA, ratio, s_alpha, s_rho = row
    X = 0.013
    Y = 2 * X if regime == "Y>X" else X / 2
    A = 1.0 if sA == "+" else -1.0
    pi, mu = (0.2, 0.4) if ratio == "<1" else (0.4, 0.2)
    alpha, w = _ctrl_one(pi, mu, A, Y, X, gamma=0.65, C=3.0)
    assert (alpha < 0) == (s_alpha == "-") and alpha != 0
    assert (w > 1) == (s_rho == ">1") and w != 1


def test_worked_values():
    # gamma=0.65, X=0.013, C=3.  Y = 2X: alpha = -0.65 for A>0 -> rho = (0.5)^-0.65
    cases = [
        (0.2, 0.4, 1, 0.026, 2 ** 0.65), (0.4, 0.2, 1, 0.026, 2 ** -0.65),
        (0.4, 0.2, -1, 0.026, 2 ** 0.65), (0.2, 0.4, -1, 0.026, 2 ** -0.65),
        (0.2, 0.4, 1, 0.0065, 2 ** -0.325), (0.4, 0.2, 1, 0.0065, 2 ** 0.325),
        (0.4, 0.2, -1, 0.0065, 2 ** -0.325), (0.2, 0.4, -1, 0.0065, 2 ** 0.325),
    ]
    for pi, mu, A, Y, want in cases:
        _, w = _ctrl_one(pi, mu, A, Y, 0.013, 0.65, 3.0)
        assert abs(w - want) < 1e-12
    assert abs(2 ** 0.65 - 1.569168) < 1e-6 and abs(2 ** 0.325 - 1.252664) < 1e-6


def test_clip_at_C():
    # pi=.01, mu=.5, Y>X, A>0: alpha=-0.65, rho = 50^0.65 = 12.7 -> clipped to C=3
    alpha, w = _ctrl_one(0.01, 0.5, 1.0, 0.026, 0.013, 0.65, 3.0)
    assert abs(alpha + 0.65) < 1e-15
    assert abs(50 ** 0.65 - 12.715) < 1e-3
    assert w == 3.0


@pytest.mark.parametrize("pi,mu,A,Y", [(0.3, 0.3, 1, 0.05), (0.2, 0.4, 0.0, 0.05),
                                       (0.2, 0.4, 1, 0.013), (0.2, 0.4, -1, 0.013)])
def test_weight_is_one_when_alpha_or_ratio_vanishes(pi, mu, A, Y):
    _, w = _ctrl_one(pi, mu, A, Y, 0.013, 0.65, 3.0)
    assert abs(w - 1.0) < 1e-15


def test_gamma_one_y_zero_is_tis():
    # alpha = 1 -> weight = min(pi/mu, C): token-level TIS (Sec. 2.2, Eq. tis_objective)
    for pi, mu in ((0.2, 0.4), (0.4, 0.2), (0.9, 0.1), (0.05, 0.06)):
        alpha, w = _ctrl_one(pi, mu, 2.5, 0.0, 0.013, 1.0, 3.0)
        assert alpha == 1.0
        assert abs(w - min(pi / mu, 3.0)) < 1e-12


def test_larger_gap_gives_stronger_correction():
    # Sec. 4.1: the update strength grows with |X - Y|
    ws = [_ctrl_one(0.2, 0.4, 1.0, Y, 0.013, 0.65, 10.0)[1] for Y in (0.014, 0.02, 0.03, 0.05)]
    assert all(b > a for a, b in zip(ws, ws[1:]))


def test_controller_levels_and_mask():
    B, L, ng = 6, 9, 2
    mask, lp_pi, lp_mu, _, _, g = _random_batch(B, L, ng, 8)
    red = oracle.discrepancy_reduce(B, L, lp_pi, lp_mu, mask, g, ng)
    adv = np.array([1.0, -1.0, 0.5, -0.5, 0.0, 2.0])
    X = red["stats"][0] * 0.5 + 1e-9
    for level, Yof in ((oracle.Y_GROUP, lambda i: red["group_y"][g[i]]),
                       (oracle.Y_SEQUENCE, lambda i: red["seq_mean_d"][i]),
                       (oracle.Y_BATCH, lambda i: red["stats"][0])):
        alpha, w = oracle.controller_step(B, L, mask, g, lp_pi, lp_mu, adv, False, level,
                                          red["seq_mean_d"], red["group_y"], red["stats"],
                                          X, 0.35, 5.0)
        alpha, w = alpha.reshape(B, L), w.reshape(B, L)
        for i in range(B):
            for j in range(L):
                if not mask[i, j]:
                    assert alpha[i, j] == 0 and w[i, j] == 0
                    continue
                a = 0.35 * np.sign(adv[i]) * (1 - Yof(i) / X)
                rho = (math.exp(lp_pi[i, j]) / math.exp(lp_mu[i, j])) ** a
                assert abs(alpha[i, j] - a) < 1e-13
                assert abs(w[i, j] - min(rho, 5.0)) < 1e-12 * max(1, rho)


def test_controller_rejects_bad_hyperparameters():
    for X, gamma, C in ((0.0, 0.5, 3.0), (0.01, 0.0, 3.0), (0.01, 0.5, 1.0), (-1, 0.5, 3)):
        with pytest.raises(ValueError):
            _ctrl_one(0.2, 0.4, 1.0, 0.02, X, gamma, C)


# ------------------------------------------------------------ controller modes
# TIS (Eq. tis_objective), MIS (Eq. mis_objective) and the two one-sided
# ablations of Sec. 5 (continuous reduction, fallback to GRPO), pinned by
# their closed forms.
def _ctrl_mode(pi, mu, A, Y, mode, k=1.0, X=0.013, gamma=0.65, C=3.0):
    alpha, w = oracle.controller_step(1, 1, np.ones(1, np.uint8), np.zeros(1, np.int32),
                                      np.log([pi]), np.log([mu]), np.array([A]), False,
                                      oracle.Y_BATCH, None, None,
                                      np.array([Y] + [0.0] * (oracle.N_STATS - 1)), X, gamma, C,
                                      mode=mode, k=k)
    return alpha[0], w[0]


@pytest.mark.parametrize("pi,mu,want", [(0.2, 0.4, 0.5), (0.4, 0.2, 2.0), (0.01, 0.5, 0.02),
                                        (0.9, 0.1, 3.0), (0.3, 0.3, 1.0)])
def test_tis_is_truncated_ratio(pi, mu, want):
    for A, Y in ((1.0, 0.026), (-1.0, 0.0065), (0.0, 0.013)):
        alpha, w = _ctrl_mode(pi, mu, A, Y, oracle.CTRL_TIS)
        assert alpha == 1.0
        assert abs(w - want) < 1e-12


def test_tis_equals_acrl_at_gamma_one_y_zero():
    for pi, mu in ((0.2, 0.4), (0.4, 0.2), (0.9, 0.1)):
        _, w_acrl = _ctrl_mode(pi, mu, 1.0, 0.0, oracle.CTRL_ACRL, gamma=1.0)
        _, w_tis = _ctrl_mode(pi, mu, 1.0, 0.0, oracle.CTRL_TIS)
        assert abs(w_acrl - w_tis) < 1e-12


def test_mis_weights_whole_sequences():
    # 3 sequences of 4 slots; token log-ratios chosen so the sequence ratios
    # are 2 (kept), 4 (> C = 3: masked to 0) and 1/2 (kept)
    B, L = 3, 4
    mask = np.array([[1, 1, 1, 1], [1, 1, 1, 0], [1, 1, 0, 0]], np.uint8)
    lp_mu = np.log(np.full((B, L), 0.3))
    lr = np.zeros((B, L))
    lr[0, :4] = [math.log(2) * f for f in (0.1, 0.2, 0.3, 0.4)]
    lr[1, :3] = [math.log(4) / 3] * 3
    lr[1, 3] = 5.0                       # a masked slot must not count
    lr[2, :2] = [-math.log(2) * 0.75, -math.log(2) * 0.25]
    lp_pi = lp_mu + lr
    adv = np.array([1.0, -1.0, 0.0])
    stats = np.zeros(oracle.N_STATS)
    alpha, w = oracle.controller_step(B, L, mask, np.zeros(B, np.int32), lp_pi, lp_mu, adv, False,
                                      oracle.Y_BATCH, None, None, stats, 0.013, 0.65, 3.0,
                                      mode=oracle.CTRL_MIS)
    w = w.reshape(B, L)
    want = [2.0, 0.0, 0.5]
    for i in range(B):
        for j in range(L):
            if mask[i, j]:
                assert abs(w[i, j] - want[i]) < 1e-12
            else:
                assert w[i, j] == 0.0


@pytest.mark.parametrize("k", [1.0, 3.0])
def test_continuous_reduction_fixed_alpha(k):
    # alpha = -k for A > 0 (quadrants I, II), +k for A < 0 (III, IV), any Y
    for Y in (0.026, 0.0065):
        a, w = _ctrl_mode(0.2, 0.4, 1.0, Y, oracle.CTRL_CONTINUOUS, k=k, C=100.0)
        assert a == -k and abs(w - 2.0 ** k) < 1e-12
        a, w = _ctrl_mode(0.4, 0.2, 1.0, Y, oracle.CTRL_CONTINUOUS, k=k, C=100.0)
        assert a == -k and abs(w - 0.5 ** k) < 1e-12
        a, w = _ctrl_mode(0.4, 0.2, -1.0, Y, oracle.CTRL_CONTINUOUS, k=k, C=100.0)
        assert a == k and abs(w - 2.0 ** k) < 1e-12
        a, w = _ctrl_mode(0.4, 0.2, 0.0, Y, oracle.CTRL_CONTINUOUS, k=k)
        assert a == 0 and w == 1.0
    # clip: 2^3 = 8 > C = 3
    assert _ctrl_mode(0.2, 0.4, 1.0, 0.02, oracle.CTRL_CONTINUOUS, k=3.0)[1] == 3.0


def test_fallback_is_grpo_below_x_and_acrl_above():
    for pi, mu, A in ((0.2, 0.4, 1.0), (0.4, 0.2, -1.0), (0.01, 0.5, 1.0)):
        a, w = _ctrl_mode(pi, mu, A, 0.0065, oracle.CTRL_FALLBACK)
        assert a == 0.0 and w == 1.0
        for Y in (0.013, 0.026):
            got = _ctrl_mode(pi, mu, A, Y, oracle.CTRL_FALLBACK)
            want = _ctrl_mode(pi, mu, A, Y, oracle.CTRL_ACRL)
            assert got == want


def test_controller_rejects_bad_mode_or_k():
    with pytest.raises(ValueError):
        _ctrl_mode(0.2, 0.4, 1.0, 0.02, 7)
    with pytest.raises(ValueError):
        _ctrl_mode(0.2, 0.4, 1.0, 0.02, oracle.CTRL_CONTINUOUS, k=0.0)


# ------------------------------------------------------------ undefined inputs
# min(rho, C) is defined for a ratio rho; an undefined ratio (a NaN log-prob,
# the scorer's mark of an invalid token id) or an undefined Y (a response
# outside every group) leaves the weight undefined: NaN, never the clip C.
@pytest.mark.parametrize("mode", [oracle.CTRL_ACRL, oracle.CTRL_TIS, oracle.CTRL_CONTINUOUS,
                                  oracle.CTRL_FALLBACK])
@pytest.mark.parametrize("A", [1.0, -1.0, 0.0])
def test_nan_logprob_gives_nan_weight(mode, A):
    # Y = 0.026 > X: FALLBACK takes the ACRL branch; A = 0 (alpha = 0) must
    # not turn the undefined ratio into 1
    a, w = _ctrl_mode(float("nan"), 0.4, A, 0.026, mode)
    assert math.isnan(w)
    a, w = _ctrl_mode(0.2, float("nan"), A, 0.026, mode)
    assert math.isnan(w)


def test_nan_logprob_mis_weights_its_sequence_nan():
    B, L = 2, 3
    mask = np.ones((B, L), np.uint8)
    lp_mu = np.log(np.full((B, L), 0.3))
    lp_pi = lp_mu.copy()
    lp_pi[0, 1] = float("nan")
    _, w = oracle.controller_step(B, L, mask, np.zeros(B, np.int32), lp_pi, lp_mu, np.ones(B), False,
                                  oracle.Y_BATCH, None, None, np.zeros(oracle.N_STATS), 0.013, 0.65, 3.0,
                                  mode=oracle.CTRL_MIS)
    w = w.reshape(B, L)
    assert np.isnan(w[0]).all() and np.all(w[1] == 1.0)


@pytest.mark.parametrize("mode", [oracle.CTRL_ACRL, oracle.CTRL_FALLBACK])
def test_group_outside_range_gives_nan(mode):
    B, L, ng = 3, 2, 2
    mask = np.ones((B, L), np.uint8)
    lp_pi = np.log(np.full((B, L), 0.2))
    lp_mu = np.log(np.full((B, L), 0.4))
    g = np.array([0, 2, -1], np.int32)  # responses 1 and 2 belong to no group
    gy = np.array([0.026, 0.026])
    alpha, w = oracle.controller_step(B, L, mask, g, lp_pi, lp_mu, np.ones(B), False, oracle.Y_GROUP, None,
                                      gy, None, 0.013, 0.65, 3.0, mode=mode, n_groups=ng)
    alpha, w = alpha.reshape(B, L), w.reshape(B, L)
    assert np.isnan(alpha[1:]).all() and np.isnan(w[1:]).all()
    # response 0: alpha = 0.65 (1 - 2) = -0.65, rho = (0.2/0.4)^-0.65 (the worked value)
    assert np.allclose(alpha[0], -0.65) and np.allclose(w[0], 1.569168, atol=1e-6)
    # masked slots stay 0 whatever the group
    mask[1, 1] = 0
    alpha, w = oracle.controller_step(B, L, mask, g, lp_pi, lp_mu, np.ones(B), False, oracle.Y_GROUP, None,
                                      gy, None, 0.013, 0.65, 3.0, mode=mode, n_groups=ng)
    assert alpha.reshape(B, L)[1, 1] == 0 and w.reshape(B, L)[1, 1] == 0
