"""GPU parity of acrl_surrogate (Eq. ACRL) and acrl_lm_head_backward with the
oracle: the per-token coefficients and the loss, then the rows of dH = dZ W and
dW = dZ^T H, dZ = coef (onehot - softmax) / tau.

Bound for the backward.  The GPU rounds dZ to bf16 (relative error at most
2^-9 per element) and accumulates the bf16 products in fp32, so an element of
dH differs from the oracle's fp64 value by at most about 2^-9 times the sum of
the magnitudes of its terms (the oracle's dh_abs / dw_abs), plus the fp32
accumulation, well inside 2^-8 of the same sum; a small absolute floor covers
elements whose terms all vanish."""
import math

import numpy as np
import pytest

import inputs
import oracle
from cases import random_bf16, workload_case
from gpu_util import down, par_map, torch_dev, up, up_bf16

pytestmark = pytest.mark.gpu

BOUND = 2.0 ** -8


def _check_rows(got, ref, ref_abs, what):
    floor = 1e-6 * max(np.abs(ref).max(), 1e-30)
    err = np.abs(got - ref)
    lim = BOUND * ref_abs + floor
    bad = np.argwhere(err > lim)
    assert bad.size == 0, "%s: %d elements outside the bound, first %s: got %g ref %g abs %g" % (
        what, len(bad), bad[0], got[tuple(bad[0])], ref[tuple(bad[0])], ref_abs[tuple(bad[0])])
    # typical agreement is far tighter than the worst-case bound
    big = np.abs(ref) > 1e-3 * np.abs(ref).max()
    if big.any():
        assert np.median(err[big] / np.abs(ref[big])) < 1e-2, what


# ------------------------------------------------------------------ surrogate
def _batch(B, L, n_groups, seed, empty=()):
    r = np.random.default_rng(seed)
    lens = r.integers(1, L + 1, size=B)
    for i in empty:
        lens[i] = 0
    mask = (np.arange(L)[None, :] < lens[:, None]).astype(np.uint8)
    lp_old = np.log(r.uniform(1e-4, 1, size=(B, L))).astype(np.float32)
    lp_new = (lp_old + r.normal(0, 0.3, size=(B, L))).astype(np.float32)
    g = np.sort(r.integers(0, n_groups, size=B)).astype(np.int32)
    return mask, lp_new, lp_old, g


@pytest.mark.parametrize("B,L,ng,empty", [(9, 23, 4, ()), (64, 4096, 8, ()), (5, 1, 2, (1,)),
                                          (12, 300, 5, (0, 4)), (130, 257, 3, ())])
@pytest.mark.parametrize("per_token,weighted,eps", [(False, True, (0.2, 0.2)), (True, True, (0.2, 0.28)),
                                                    (False, False, (0.1, 0.3))])
def test_surrogate_matches_oracle(B, L, ng, empty, per_token, weighted, eps):
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    mask, lp_new, lp_old, g = _batch(B, L, ng, 7 * B + L, empty)
    r = np.random.default_rng(B + L)
    adv = r.normal(size=B * L if per_token else B).astype(np.float32)
    adv[:2] = 0.0
    wt = r.uniform(0.3, 3.0, size=B * L).astype(np.float32) if weighted else None
    t = lambda a: up(torch, dev, np.ascontiguousarray(a).reshape(-1))
    coef, loss = acrl.acrl_surrogate(B, L, ng, t(mask), up(torch, dev, g), t(lp_new), t(lp_old), t(adv),
                                     per_token, eps_low=eps[0], eps_high=eps[1],
                                     weight=None if wt is None else t(wt))
    torch.cuda.synchronize()
    # the ABI takes eps as fp32: the oracle gets the same values
    e32 = [float(np.float32(e)) for e in eps]
    rc, rl = oracle.surrogate(B, L, mask, g, ng, lp_new, lp_old, adv, adv_per_token=per_token, weight=wt,
                              eps_low=e32[0], eps_high=e32[1])
    # same fp32 inputs, fp64 on both sides: the coefficients agree to their
    # one fp32 rounding, the loss to fp64 summation order
    np.testing.assert_allclose(down(coef), rc.astype(np.float32), rtol=2e-7, atol=0)
    assert float(down(loss)[0]) == pytest.approx(rl, rel=1e-12, abs=1e-300)
    assert np.all(down(coef)[mask.reshape(-1) == 0] == 0)


def test_surrogate_empty_batch():
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    B, L, ng = 3, 8, 2
    mask = np.zeros((B, L), np.uint8)
    z = np.zeros(B * L, np.float32)
    coef, loss = acrl.acrl_surrogate(B, L, ng, up(torch, dev, mask.reshape(-1)),
                                     up(torch, dev, np.array([0, 1, 1], np.int32)), up(torch, dev, z),
                                     up(torch, dev, z), up(torch, dev, np.ones(B, np.float32)), False)
    torch.cuda.synchronize()
    assert float(down(loss)[0]) == 0.0 and np.all(down(coef) == 0)


# ------------------------------------------------------------------ backward
def _backward_case(T, V, d, seed, tau=1.0, masked=0.25):
    r = np.random.default_rng(seed)
    H = random_bf16((T, d), seed)
    W = random_bf16((V, d), seed + 1, std=2.5 / math.sqrt(d))
    ids = r.integers(0, V, size=T).astype(np.int32)
    coef = (r.normal(size=T) * 1e-2).astype(np.float32)
    coef[r.uniform(size=T) < masked] = 0.0
    coef[0] = 0.02  # at least one live row
    # the oracle's own lse of pi (natural units) for the GPU input
    lse = np.array([oracle.token_stats(oracle.logits_pi(H[t], W, 1.0 / tau), int(ids[t]))[0]
                    for t in range(T)], np.float32)
    return H, W, ids, coef, lse


def _gpu_backward(H, W, ids, coef, lse, tau, **kw):
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    dh, dw = acrl.acrl_lm_head_backward(up_bf16(torch, dev, H), up_bf16(torch, dev, W), up(torch, dev, ids),
                                        up(torch, dev, coef), up(torch, dev, lse), inv_temperature=1.0 / tau,
                                        **kw)
    torch.cuda.synchronize()
    return (None if dh is None else down(dh)), (None if dw is None else down(dw))


@pytest.mark.parametrize("T,V,d,tau", [(300, 1000, 256, 1.0), (256, 2048, 256, 1.0), (513, 300, 128, 1.0),
                                       (1, 100, 128, 1.0), (260, 4128, 384, 0.7), (77, 1100, 256, 0.7)])
def test_backward_matches_oracle(T, V, d, tau):
    H, W, ids, coef, lse = _backward_case(T, V, d, T + V + d, tau)
    dh, dw = _gpu_backward(H, W, ids, coef, lse, tau)
    rdh, rdw, rdha, rdwa = oracle.lm_head_backward(H, W, ids, coef.astype(np.float64), 1.0 / tau, want_abs=True)
    _check_rows(dh, rdh, rdha, "dH")
    _check_rows(dw, rdw, rdwa, "dW")
    # masked rows (coef 0) have no gradient
    assert np.all(dh[coef == 0] == 0)


def test_backward_chunks_accumulate_and_parts():
    T, V, d, tau = 700, 1000, 256, 1.0
    H, W, ids, coef, lse = _backward_case(T, V, d, 11, tau)
    dh, dw = _gpu_backward(H, W, ids, coef, lse, tau)
    # passes of 256 rows: dH identical (each row is one pass's), dW to fp32 order
    dh2, dw2 = _gpu_backward(H, W, ids, coef, lse, tau, token_chunk=256)
    assert np.array_equal(dh, dh2)
    np.testing.assert_allclose(dw2, dw, rtol=1e-5, atol=1e-6 * np.abs(dw).max())
    # dh only / dw only
    dh3, none = _gpu_backward(H, W, ids, coef, lse, tau, want_dw=False)
    assert none is None and np.array_equal(dh3, dh)
    none, dw3 = _gpu_backward(H, W, ids, coef, lse, tau, want_dh=False)
    assert none is None and np.array_equal(dw3, dw)
    # accumulate: two calls over halves add up to the whole
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    Wd = up_bf16(torch, dev, W)
    acc = torch.zeros((V, d), dtype=torch.float32, device=dev)
    for a, b in ((0, 300), (300, T)):
        acrl.acrl_lm_head_backward(up_bf16(torch, dev, H[a:b]), Wd, up(torch, dev, ids[a:b]),
                                   up(torch, dev, coef[a:b]), up(torch, dev, lse[a:b]), want_dh=False,
                                   dw=acc, accumulate_dw=True)
    torch.cuda.synchronize()
    np.testing.assert_allclose(down(acc), dw, rtol=1e-5, atol=1e-6 * np.abs(dw).max())


def test_backward_slot_map_and_empty():
    T, V, d, tau = 300, 1000, 256, 1.0
    H, W, ids, coef, lse = _backward_case(T, V, d, 12, tau)
    dh, dw = _gpu_backward(H, W, ids, coef, lse, tau)
    # the same coefficients and lse scattered to slots through row_slot
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    n_slots = 2 * T + 5
    slots = np.random.default_rng(3).permutation(n_slots)[:T].astype(np.int32)
    cs = np.full(n_slots, np.nan, np.float32)
    ls = np.full(n_slots, np.nan, np.float32)
    cs[slots], ls[slots] = coef, lse
    dh2, dw2 = acrl.acrl_lm_head_backward(up_bf16(torch, dev, H), up_bf16(torch, dev, W), up(torch, dev, ids),
                                          up(torch, dev, cs), up(torch, dev, ls), row_slot=up(torch, dev, slots))
    torch.cuda.synchronize()
    assert np.array_equal(down(dh2), dh) and np.array_equal(down(dw2), dw)
    # no rows: dW = 0 (or untouched when accumulating)
    e = np.zeros((0, d), np.uint16)
    dwz = torch.full((V, d), 7.0, dtype=torch.float32, device=dev)
    acrl.acrl_lm_head_backward(up_bf16(torch, dev, e), up_bf16(torch, dev, W), up(torch, dev, np.zeros(0, np.int32)),
                               up(torch, dev, np.zeros(1, np.float32)), up(torch, dev, np.zeros(1, np.float32)),
                               want_dh=False, dw=dwz)
    torch.cuda.synchronize()
    assert np.all(down(dwz) == 0)


def test_backward_full_size_sampled_rows():
    """d = 4096, V = 151936 in the bench's launch configuration (16384-row
    passes, a ragged second pass).  40 rows carry a coefficient -- both ends
    of each pass, of a 256-row tile and of a 2048-row block of tiles, one row
    in every block, the rest seeded -- so every dW row is a sum over those
    tokens and the oracle can form it; dH is checked on rows with and without
    a coefficient."""
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    w = inputs.WORKLOADS["q8b"]
    T, d, V = 16384 + 300, w.d, w.V
    Hd = inputs.hidden_bf16_torch(w, T, dev)
    Wd = inputs.weights_bf16_torch(w, dev)
    r = np.random.default_rng(8)
    edges = [0, 255, 256, 2047, 2048, 16383, 16384, 16385, T - 1]  # T - 1: the ragged tail pass
    blocks = [b * 2048 + 700 for b in range(1, 8)]
    rest = r.choice(np.setdiff1d(np.arange(T), edges + blocks), size=40 - len(edges) - len(blocks), replace=False)
    live = np.sort(np.concatenate([edges, blocks, rest]))
    ids = r.integers(0, V, size=T).astype(np.int32)
    coef = np.zeros(T, np.float32)
    coef[live] = r.normal(size=live.size).astype(np.float32) * 1e-3
    Hl = down(Hd[torch.from_numpy(live).to(dev)].view(torch.int16)).view(np.uint16)
    Wh = down(Wd.view(torch.int16)).view(np.uint16)
    lse = np.zeros(T, np.float32)
    oracle.lib()
    lse[live] = par_map(lambda kt: oracle.token_stats(oracle.logits_pi(Hl[kt[0]], Wh, 1.0), int(ids[kt[1]]))[0],
                        enumerate(live))
    dh, dw = acrl.acrl_lm_head_backward(Hd, Wd, up(torch, dev, ids), up(torch, dev, coef), up(torch, dev, lse))
    torch.cuda.synchronize()
    wrows = np.concatenate([np.unique(ids[live]), r.choice(V, size=6, replace=False), [V - 1]])
    rdh, rdw, rdha, rdwa = oracle.lm_head_backward(Hl, Wh, ids[live], coef[live].astype(np.float64), 1.0,
                                                   wrows=wrows, want_abs=True)
    _check_rows(down(dh[torch.from_numpy(live).to(dev)]), rdh, rdha, "dH (full size)")
    _check_rows(down(dw[torch.from_numpy(wrows).to(dev)]), rdw, rdwa, "dW (full size)")
    dead = np.setdiff1d(np.arange(0, T, 997), live)
    assert np.all(down(dh[torch.from_numpy(dead).to(dev)]) == 0)


@pytest.mark.parametrize("name", ["q17b", "mx"])
def test_backward_other_heads_sampled_rows(name):
    """The 1.7B-shaped head (d = 2048) and the d = 5120 head at tau = 0.7,
    V = 151936: 4096 + 300 rows in passes of 2048 (three passes, the last
    ragged).  24 rows carry a coefficient -- both ends of the call, of each
    pass and of a tile, the rest seeded -- and the oracle forms dH on them
    and dW on the rows they touch and a few others."""
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    w = inputs.WORKLOADS[name]
    tau = 1.0 / w.inv_temperature
    T, d, V = 4096 + 300, w.d, w.V
    Hd = inputs.hidden_bf16_torch(w, T, dev)
    Wd = inputs.weights_bf16_torch(w, dev)
    r = np.random.default_rng(9)
    edges = [0, 255, 256, 2047, 2048, 4095, 4096, T - 1]
    rest = r.choice(np.setdiff1d(np.arange(T), edges), size=24 - len(edges), replace=False)
    live = np.sort(np.concatenate([edges, rest]))
    ids = r.integers(0, V, size=T).astype(np.int32)
    coef = np.zeros(T, np.float32)
    coef[live] = r.normal(size=live.size).astype(np.float32) * 1e-3
    Hl = down(Hd[torch.from_numpy(live).to(dev)].view(torch.int16)).view(np.uint16)
    Wh = down(Wd.view(torch.int16)).view(np.uint16)
    lse = np.zeros(T, np.float32)
    oracle.lib()
    lse[live] = par_map(lambda kt: oracle.token_stats(oracle.logits_pi(Hl[kt[0]], Wh, 1.0 / tau),
                                                      int(ids[kt[1]]))[0], enumerate(live))
    dh, dw = acrl.acrl_lm_head_backward(Hd, Wd, up(torch, dev, ids), up(torch, dev, coef), up(torch, dev, lse),
                                        inv_temperature=1.0 / tau, token_chunk=2048)
    torch.cuda.synchronize()
    wrows = np.concatenate([np.unique(ids[live]), r.choice(V, size=6, replace=False), [V - 1]])
    rdh, rdw, rdha, rdwa = oracle.lm_head_backward(Hl, Wh, ids[live], coef[live].astype(np.float64), 1.0 / tau,
                                                   wrows=wrows, want_abs=True)
    _check_rows(down(dh[torch.from_numpy(live).to(dev)]), rdh, rdha, "dH (%s)" % name)
    _check_rows(down(dw[torch.from_numpy(wrows).to(dev)]), rdw, rdwa, "dW (%s)" % name)
    dead = np.setdiff1d(np.arange(0, T, 331), live)
    assert np.all(down(dh[torch.from_numpy(dead).to(dev)]) == 0)


def test_chain_score_surrogate_backward_small_workload():
    """The small workload end to end: the GPU's own log-probs and lse feed its
    surrogate and backward; the oracle runs its own chain on the same inputs.
    The coefficients then differ by the log-prob tolerance (relative 2e-3 at
    most: coef is proportional to exp(logp_new)), so dH and dW agree within
    that on top of the bf16 bound (no token sits near a clip edge)."""
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    c = workload_case("tiny")
    w = c["w"]
    T = c["H"].shape[0]
    r = np.random.default_rng(9)
    old_shift = r.normal(0, 0.01, size=T)  # r_t within 3% of 1: far from the 0.8 / 1.2 clip edges
    Hd, Wd = up_bf16(torch, dev, c["H"]), up_bf16(torch, dev, c["W"])
    hq, hs = acrl.acrl_quantize_fp8(Hd, w.scaling)
    wq, ws = acrl.acrl_quantize_fp8(Wd, w.scaling)
    ids = up(torch, dev, c["ids"])
    sc = acrl.acrl_score_pi_mu(Hd, Wd, hq, hs, wq, ws, w.scaling, ids, inv_temperature=w.inv_temperature,
                               out_slot=up(torch, dev, c["slots"]), n_slots=w.slots)
    mask = up(torch, dev, c["mask"].reshape(-1))
    groups = up(torch, dev, c["groups"])
    # logp_old: the slots' pi log-probs (oracle) shifted by a seeded amount
    ref = oracle.score(c["H"], c["W"], c["hq"], c["hs"], c["wq"], c["ws"], w.scaling, c["ids"],
                       inv_temperature=w.inv_temperature)
    lp_old = np.zeros(w.slots, np.float32)
    lp_old[c["slots"]] = (ref["logp_pi"] + old_shift).astype(np.float32)
    adv = c["adv"].astype(np.float32)
    coef, loss = acrl.acrl_surrogate(w.B, w.L, w.n_prompts, mask, groups, sc["logp_pi"], up(torch, dev, lp_old),
                                     up(torch, dev, adv), False)
    dh, dw = acrl.acrl_lm_head_backward(Hd, Wd, ids, coef, sc["lse_pi"], inv_temperature=w.inv_temperature,
                                        row_slot=up(torch, dev, c["slots"]))
    torch.cuda.synchronize()
    lp_new_o = np.zeros(w.slots)
    lp_new_o[c["slots"]] = ref["logp_pi"]
    e32 = float(np.float32(0.2))
    rc, rl = oracle.surrogate(w.B, w.L, c["mask"], c["groups"], w.n_prompts, lp_new_o, lp_old, adv,
                              eps_low=e32, eps_high=e32)
    assert float(down(loss)[0]) == pytest.approx(rl, rel=3e-3)
    rdh, rdw, rdha, rdwa = oracle.lm_head_backward(c["H"], c["W"], c["ids"], rc[c["slots"]], w.inv_temperature,
                                                   want_abs=True)
    for got, want, mag, what in ((down(dh), rdh, rdha, "dH"), (down(dw), rdw, rdwa, "dW")):
        err = np.abs(got - want)
        assert np.all(err <= BOUND * mag + 3e-3 * np.abs(want) + 1e-6 * np.abs(want).max()), what
