"""GPU parity of acrl_discrepancy_reduce and acrl_controller_step with the
oracle, fed the same per-token log-probs, plus the small workload end to end
(quantize -> score -> reduce -> controller) against the oracle's whole chain."""
import math

import numpy as np
import pytest

import inputs
import oracle
from cases import TOL_LOGP, tol_seq_logratio, workload_case
from gpu_util import down, torch_dev, up, up_bf16

pytestmark = pytest.mark.gpu


def _batch(B, L, n_groups, seed, empty=(), shuffle=False):
    r = np.random.default_rng(seed)
    lens = r.integers(1, L + 1, size=B)
    for i in empty:
        lens[i] = 0
    mask = (np.arange(L)[None, :] < lens[:, None]).astype(np.uint8)
    lp_pi = np.log(r.uniform(1e-5, 1, size=(B, L))).astype(np.float32)
    lp_mu = np.minimum(lp_pi + r.normal(0, 0.1, size=(B, L)), 0).astype(np.float32)
    ent_pi = r.uniform(0, 9, size=(B, L)).astype(np.float32)
    ent_mu = r.uniform(0, 9, size=(B, L)).astype(np.float32)
    g = np.sort(r.integers(0, n_groups, size=B)).astype(np.int32)
    if shuffle:  # responses of a group scattered over the batch
        g = r.permutation(g).astype(np.int32)
    return mask, lp_pi, lp_mu, ent_pi, ent_mu, g


def _gpu_reduce(B, L, ng, mask, lp_pi, lp_mu, ent_pi, ent_mu, g):
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    t = lambda a: up(torch, dev, np.ascontiguousarray(a).reshape(-1))
    out = acrl.acrl_discrepancy_reduce(B, L, ng, t(lp_pi), t(lp_mu), t(mask), up(torch, dev, g),
                                       entropy_pi=t(ent_pi), entropy_mu=t(ent_mu))
    torch.cuda.synchronize()
    return {k: down(v) for k, v in out.items() if v is not None and not k.startswith("_")}


@pytest.mark.parametrize("B,L,ng,empty,shuffle", [
    (9, 23, 4, (), False), (64, 4096, 8, (), False), (5, 1, 2, (1,), False), (1, 700, 1, (), False),
    (12, 300, 5, (0, 4), False), (130, 257, 3, (), False), (3, 16, 8, (), False),
    (9, 23, 4, (), True), (130, 257, 3, (), True), (12, 300, 5, (0, 4), True),
    (3000, 32, 1500, (5, 17), False), (3000, 32, 1500, (5, 17), True)])
def test_reduce_matches_oracle(B, L, ng, empty, shuffle):
    # sorted group ids take the binary-search path of the group kernel,
    # shuffled ones the scan; groups with no response and > 1024 groups too
    mask, lp_pi, lp_mu, ent_pi, ent_mu, g = _batch(B, L, ng, B * L, empty, shuffle)
    got = _gpu_reduce(B, L, ng, mask, lp_pi, lp_mu, ent_pi, ent_mu, g)
    ref = oracle.discrepancy_reduce(B, L, lp_pi, lp_mu, mask, g, ng, ent_pi, ent_mu)
    # same fp32 inputs, both sides accumulate in fp64: agreement to rounding
    assert np.array_equal(got["seq_len"], ref["seq_len"])
    np.testing.assert_allclose(got["seq_sum_d"], ref["seq_sum_d"], rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(got["seq_sum_logratio"], ref["seq_sum_logratio"], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(got["seq_mean_d"], ref["seq_mean_d"].astype(np.float32), rtol=1e-6, atol=0)
    np.testing.assert_allclose(got["group_y"], ref["group_y"].astype(np.float32), rtol=1e-6, atol=0)
    assert np.array_equal(got["group_nseq"], ref["group_nseq"])
    np.testing.assert_allclose(got["stats"], ref["stats"], rtol=1e-10, atol=1e-15)
    np.testing.assert_allclose(got["d_tok"], ref["d_tok"].astype(np.float32), rtol=1e-6, atol=0)


def test_reduce_deterministic():
    B, L, ng = 64, 2048, 8
    args = _batch(B, L, ng, 3)
    a = _gpu_reduce(B, L, ng, *args)
    b = _gpu_reduce(B, L, ng, *args)
    for k in a:
        assert np.array_equal(a[k], b[k]), k


def _oracle_y(B, L, ng, mask, lp_pi, lp_mu, g):
    """The discrepancy levels Y (and X) that both controllers take as inputs:
    the oracle's reduce of the seeded batch, in the ABI's types."""
    ref = oracle.discrepancy_reduce(B, L, lp_pi, lp_mu, mask, g, ng)
    return {"seq_mean_d": ref["seq_mean_d"].astype(np.float32), "group_y": ref["group_y"].astype(np.float32),
            "stats": ref["stats"].astype(np.float64), "seq_sum_logratio": ref["seq_sum_logratio"]}


@pytest.mark.parametrize("level", [oracle.Y_GROUP, oracle.Y_SEQUENCE, oracle.Y_BATCH])
@pytest.mark.parametrize("per_token", [False, True])
def test_controller_matches_oracle(level, per_token):
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    B, L, ng = 24, 300, 3
    mask, lp_pi, lp_mu, ent_pi, ent_mu, g = _batch(B, L, ng, 21)
    red = _oracle_y(B, L, ng, mask, lp_pi, lp_mu, g)
    r = np.random.default_rng(22)
    adv = (r.normal(size=B * L if per_token else B)).astype(np.float32)
    adv[:3] = 0.0
    for X, gamma, C in ((float(red["stats"][0]) * 0.5, 0.65, 3.0), (float(red["stats"][0]) * 2, 0.35, 5.0)):
        t = lambda a: up(torch, dev, np.ascontiguousarray(a).reshape(-1))
        alpha, weight = acrl.acrl_controller_step(
            B, L, ng, t(mask), up(torch, dev, g), t(lp_pi), t(lp_mu), t(adv), per_token, level,
            t(red["seq_mean_d"]), t(red["group_y"]), t(red["stats"]), X, gamma, C)
        torch.cuda.synchronize()
        a_ref, w_ref = oracle.controller_step(B, L, mask, g, lp_pi, lp_mu, adv, per_token, level,
                                              red["seq_mean_d"], red["group_y"], red["stats"],
                                              float(np.float32(X)), float(np.float32(gamma)),
                                              float(np.float32(C)))
        # fp64 on both sides from identical fp32 inputs, one final fp32 rounding
        np.testing.assert_allclose(down(alpha), a_ref.astype(np.float32), rtol=2 ** -23, atol=1e-30)
        np.testing.assert_allclose(down(weight), w_ref.astype(np.float32), rtol=2 ** -23, atol=1e-30)
        assert np.all(down(weight)[mask.reshape(-1) == 0] == 0)
        assert np.all(down(weight) <= np.float32(C))


@pytest.mark.parametrize("mode,k", [(oracle.CTRL_TIS, 1.0), (oracle.CTRL_MIS, 1.0),
                                    (oracle.CTRL_CONTINUOUS, 1.0), (oracle.CTRL_CONTINUOUS, 3.0),
                                    (oracle.CTRL_FALLBACK, 1.0)])
def test_controller_modes_match_oracle(mode, k):
    # TIS (Eq. tis_objective), MIS (Eq. mis_objective), and the continuous-
    # reduction / fallback-to-GRPO ablations of Sec. 5
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    B, L, ng = 24, 300, 3
    mask, lp_pi, lp_mu, ent_pi, ent_mu, g = _batch(B, L, ng, 31)
    red = _oracle_y(B, L, ng, mask, lp_pi, lp_mu, g)
    adv = np.random.default_rng(32).normal(size=B).astype(np.float32)
    adv[:2] = 0.0
    t = lambda a: up(torch, dev, np.ascontiguousarray(a).reshape(-1))
    C = 3.0
    # MIS keeps a sequence iff its ratio is <= C: leave out sequences whose
    # log-ratio sum lies within rounding of ln C (none for this seed)
    near = np.abs(red["seq_sum_logratio"] - math.log(C)) < 1e-6
    assert not near.any()
    for X in (float(red["stats"][0]) * 0.5, float(red["stats"][0]) * 2):
        alpha, weight = acrl.acrl_controller_step(
            B, L, ng, t(mask), up(torch, dev, g), t(lp_pi), t(lp_mu), t(adv), False, oracle.Y_GROUP,
            t(red["seq_mean_d"]), t(red["group_y"]), t(red["stats"]), X, 0.65, C, mode=mode, k=k,
            seq_sum_logratio=up(torch, dev, red["seq_sum_logratio"]))
        torch.cuda.synchronize()
        a_ref, w_ref = oracle.controller_step(B, L, mask, g, lp_pi, lp_mu, adv, False, oracle.Y_GROUP,
                                              red["seq_mean_d"], red["group_y"], red["stats"],
                                              float(np.float32(X)), float(np.float32(0.65)), C,
                                              mode=mode, k=float(np.float32(k)))
        np.testing.assert_allclose(down(alpha), a_ref.astype(np.float32), rtol=2 ** -23, atol=1e-30)
        # MIS: the GPU sums the fp32 log-ratios in its own order (fp64), the
        # oracle multiplies the token ratios; elsewhere both round once
        rtol = 1e-9 * L if mode == oracle.CTRL_MIS else 2 ** -23
        np.testing.assert_allclose(down(weight), w_ref.astype(np.float32), rtol=max(rtol, 2 ** -23),
                                   atol=1e-30)
        assert np.all(down(weight)[mask.reshape(-1) == 0] == 0)
        if mode == oracle.CTRL_MIS:
            kept = (red["seq_sum_logratio"] <= math.log(C)).sum()
            assert 0 < kept < B  # both branches exercised


def test_small_workload_end_to_end():
    """quantize -> score -> reduce -> controller on the device against the
    oracle's whole chain on the same seeded inputs."""
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    c = workload_case("tiny")
    w = c["w"]
    h = up_bf16(torch, dev, c["H"])
    W = up_bf16(torch, dev, c["W"])
    hq, hs = acrl.acrl_quantize_fp8(h, w.scaling)
    wq, ws = acrl.acrl_quantize_fp8(W, w.scaling)
    slots = up(torch, dev, c["slots"])
    sc = acrl.acrl_score_pi_mu(h, W, hq, hs, wq, ws, w.scaling, up(torch, dev, c["ids"]),
                               inv_temperature=w.inv_temperature, out_slot=slots, n_slots=w.slots)
    m = up(torch, dev, c["mask"].reshape(-1))
    g = up(torch, dev, c["groups"])
    red = acrl.acrl_discrepancy_reduce(w.B, w.L, w.n_prompts, sc["logp_pi"], sc["logp_mu"], m, g,
                                       entropy_pi=sc["entropy_pi"], entropy_mu=sc["entropy_mu"])
    torch.cuda.synchronize()
    # oracle chain (its own quantization, scores and reduce)
    sref = oracle.score(c["H"], c["W"], c["hq"], c["hs"], c["wq"], c["ws"], w.scaling, c["ids"],
                        inv_temperature=w.inv_temperature)
    lp_pi = np.zeros(w.slots)
    lp_mu = np.zeros(w.slots)
    lp_pi[c["slots"]] = sref["logp_pi"]
    lp_mu[c["slots"]] = sref["logp_mu"]
    rref = oracle.discrepancy_reduce(w.B, w.L, lp_pi, lp_mu, c["mask"], c["groups"], w.n_prompts)
    # the threshold X is taken from the oracle chain and handed to both sides
    X = float(rref["stats"][0]) * 0.5
    alpha, weight = acrl.acrl_controller_step(w.B, w.L, w.n_prompts, m, g, sc["logp_pi"], sc["logp_mu"],
                                              up(torch, dev, c["adv"]), False, acrl.Y_GROUP,
                                              red["seq_mean_d"], red["group_y"], red["stats"],
                                              X, 0.65, 3.0)
    torch.cuda.synchronize()
    gl = down(sc["logp_pi"])
    assert np.abs(gl - lp_pi).max() <= TOL_LOGP
    assert np.abs(down(sc["logp_mu"]) - lp_mu).max() <= TOL_LOGP
    n = rref["seq_len"]
    dsl = np.abs(down(red["seq_sum_logratio"]) - rref["seq_sum_logratio"])
    assert np.all(dsl <= np.array([1e-3 * math.sqrt(max(k, 1)) for k in n])), dsl
    assert np.array_equal(down(red["seq_len"]), n)
    # discrepancies: d = |pi - mu| of probabilities differ by at most |dp| <~ p*|dlogp|
    assert abs(float(down(red["stats"])[0]) - rref["stats"][0]) <= 1e-3 * max(rref["stats"][0], 1e-6) + 1e-6
    # controller fed the oracle chain's own Y agrees with the device weights
    a_ref, w_ref = oracle.controller_step(w.B, w.L, c["mask"], c["groups"], lp_pi, lp_mu, c["adv"], False,
                                          oracle.Y_GROUP, rref["seq_mean_d"], rref["group_y"],
                                          rref["stats"], X, 0.65, 3.0)
    wg = down(weight)
    # weight = exp(alpha * log-ratio): |dw| <= w * |alpha| * 2 * TOL_LOGP (+ Y differences)
    assert np.all(np.abs(wg - w_ref) <= wg * (0.65 * 3 * 2 * TOL_LOGP + 1e-3) + 1e-6)


@pytest.mark.parametrize("B,L,ng", [(0, 16, 0), (0, 16, 3), (4, 16, 2), (3, 0, 2)])
def test_reduce_empty_and_all_masked(B, L, ng):
    # degenerate batches: no responses, no slots, or every slot masked
    # (n_i = 0 everywhere): every output the oracle gives, zeros throughout
    mask = np.zeros((B, L), np.uint8)
    lp = np.log(np.full((B, L), 0.5)).astype(np.float32)
    g = (np.arange(B) % max(ng, 1)).astype(np.int32)
    got = _gpu_reduce(B, L, ng, mask, lp, lp - 0.1, lp * 0, lp * 0, g)
    ref = oracle.discrepancy_reduce(B, L, lp, lp - 0.1, mask, g, ng)
    assert np.array_equal(got["seq_len"], ref["seq_len"])
    assert np.array_equal(got["stats"], ref["stats"])
    assert np.array_equal(got["group_y"], ref["group_y"].astype(np.float32))
    assert np.array_equal(got["seq_mean_d"], ref["seq_mean_d"].astype(np.float32))
    assert np.array_equal(got["group_nseq"], ref["group_nseq"])
    if B * L:
        assert np.all(got["d_tok"] == 0)


@pytest.mark.parametrize("mode", [oracle.CTRL_ACRL, oracle.CTRL_TIS, oracle.CTRL_MIS, oracle.CTRL_CONTINUOUS,
                                  oracle.CTRL_FALLBACK])
def test_controller_undefined_inputs_give_nan(mode):
    # a NaN log-prob in a valid slot (the scorer's mark of an invalid token id)
    # and responses whose group id lies outside [0, n_groups): weight NaN on
    # both sides (never the clip C), masked slots 0, the rest as the oracle
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    B, L, ng = 8, 40, 3
    mask, lp_pi, lp_mu, _, _, g = _batch(B, L, ng, 41)
    mask[:, 0] = 1
    lp_pi[2, 0] = np.nan
    lp_mu[5, 0] = np.nan
    red = _oracle_y(B, L, ng, mask, np.nan_to_num(lp_pi), np.nan_to_num(lp_mu), g)
    red["seq_sum_logratio"] = np.where(np.isnan(lp_pi - lp_mu).any(axis=1), np.nan, red["seq_sum_logratio"])
    g = g.copy()
    g[6], g[7] = ng, -1
    adv = np.random.default_rng(42).normal(size=B).astype(np.float32)
    adv[2] = 0.0  # alpha = 0 must not turn the undefined ratio into 1
    X = float(red["stats"][0]) * 0.5
    t = lambda a: up(torch, dev, np.ascontiguousarray(a).reshape(-1))
    alpha, weight = acrl.acrl_controller_step(
        B, L, ng, t(mask), up(torch, dev, g), t(lp_pi), t(lp_mu), t(adv), False, oracle.Y_GROUP,
        t(red["seq_mean_d"]), t(red["group_y"]), t(red["stats"]), X, 0.65, 3.0, mode=mode, k=1.0,
        seq_sum_logratio=up(torch, dev, red["seq_sum_logratio"]))
    torch.cuda.synchronize()
    a_ref, w_ref = oracle.controller_step(B, L, mask, g, lp_pi, lp_mu, adv, False, oracle.Y_GROUP,
                                          red["seq_mean_d"], red["group_y"], red["stats"],
                                          float(np.float32(X)), float(np.float32(0.65)), 3.0, mode=mode,
                                          k=1.0, n_groups=ng)
    wg, ag = down(weight).reshape(B, L), down(alpha).reshape(B, L)
    assert np.array_equal(np.isnan(wg), np.isnan(w_ref.reshape(B, L)))
    assert np.array_equal(np.isnan(ag), np.isnan(a_ref.reshape(B, L)))
    assert np.isnan(wg[2, 0]) and np.isnan(wg[5, 0])
    if mode in (oracle.CTRL_ACRL, oracle.CTRL_FALLBACK):
        on = mask[6:].astype(bool)
        assert np.isnan(wg[6:][on]).all() and np.isnan(ag[6:][on]).all()
    assert np.all(wg[mask == 0] == 0)
    rtol = 1e-9 * L if mode == oracle.CTRL_MIS else 2 ** -23
    np.testing.assert_allclose(wg, w_ref.reshape(B, L).astype(np.float32), rtol=max(rtol, 2 ** -23), atol=1e-30,
                               equal_nan=True)
    np.testing.assert_allclose(ag, a_ref.reshape(B, L).astype(np.float32), rtol=2 ** -23, atol=1e-30,
                               equal_nan=True)
