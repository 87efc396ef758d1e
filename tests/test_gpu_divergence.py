"""GPU parity of the full-vocabulary measures of acrl_score_pi_mu (KL in
both directions and the Euclidean distance between softmax(z_pi) and
softmax(z_mu)) with the oracle.

Bound.  If every GPU logit is within delta of the exact one, then to first
order (the changes of the lse are p- resp. q-weighted means of the logit
changes): |dKL| <= 2 delta |p - q|_1 <= 2 delta sqrt(2 KL) (Pinsker), and
|dL2| <= |p (dz_pi - E_p dz_pi)|_2 + |q (dz_mu - E_q dz_mu)|_2
      <= 2 delta (|p|_2 + |q|_2).
The pi logits (BF16 MFMA, fp32 accumulation) are within ~1e-6 of the exact
sums at these shapes; the mu logits come from the FP8 MFMA, whose sums of
exact e4m3 products land up to ~1.6e-4 from the exact value at d = 256
(the logit_mu output against the oracle's z_mu), growing like sqrt(d): so
delta = 2e-4 sqrt(d / 256), and 1e-6 absolute for the final fp32 sums."""
import math

import numpy as np
import pytest
from scipy.special import softmax

import inputs
import oracle
from cases import lossless_integer_case, random_bf16
from gpu_util import down, par_map, torch_dev, up, up_bf16

pytestmark = pytest.mark.gpu


def _norms(H, W, hq, hs, wq, ws, scaling, tau, rows):
    """|p|_2 and |q|_2 of the rows, from the oracle's logits."""
    oracle.lib()

    def one(r):
        zp = oracle.logits_pi(H[r], W, 1.0 / tau)
        zm = oracle.logits_mu(hq[r], oracle._row_scale(hs, scaling, r), wq, ws, scaling, 1.0 / tau)
        return np.linalg.norm(softmax(zp)), np.linalg.norm(softmax(zm))

    nrm = np.array(par_map(one, rows)).reshape(-1, 2)
    return nrm[:, 0], nrm[:, 1]


def _case(T, V, d, scaling, seed):
    H = random_bf16((T, d), seed)
    W = random_bf16((V, d), seed + 1, std=2.5 / math.sqrt(d))
    hq, hs = oracle.quantize_fp8(H, scaling)
    wq, ws = oracle.quantize_fp8(W, scaling)
    ids = np.random.default_rng(seed).integers(0, V, size=T).astype(np.int32)
    return H, W, hq, hs, wq, ws, ids


def _gpu(H, W, hq, hs, wq, ws, scaling, ids, tau, **kw):
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    out = acrl.acrl_score_pi_mu(up_bf16(torch, dev, H), up_bf16(torch, dev, W), up(torch, dev, hq),
                                up(torch, dev, hs), up(torch, dev, wq), up(torch, dev, ws), scaling,
                                up(torch, dev, ids), inv_temperature=1.0 / tau, divergence=True, **kw)
    torch.cuda.synchronize()
    return {k: down(v) for k, v in out.items()}


def _check(got, ref, d, norms, rows=None, tau=1.0):
    sel = slice(None) if rows is None else rows
    delta = 2e-4 * math.sqrt(d / 256.0) / tau  # the logits carry 1/tau
    np_, nq = norms
    for k in ("kl_pi_mu", "kl_mu_pi", "l2"):
        g, r = got[k][sel], ref[k]
        if k == "l2":
            tol = 1e-6 + 2 * delta * (np_ + nq)
        else:
            tol = 1e-6 + 2 * delta * np.sqrt(2 * np.abs(r))
        err = np.abs(g - r)
        assert np.all(err <= tol), "%s: max err %g at %d (got %g, ref %g, tol %g)" % (
            k, err.max(), err.argmax(), g[err.argmax()], r[err.argmax()], tol[err.argmax()])


@pytest.mark.parametrize("T,V,d,scaling,tau", [
    (300, 1000, 256, oracle.PER_ROW, 1.0), (256, 2048, 256, oracle.PER_TENSOR, 1.0),
    (513, 300, 128, oracle.MX32, 0.7), (1, 100, 128, oracle.PER_ROW, 1.0),
    (77, 4128, 384, oracle.PER_TENSOR, 0.7), (130, 1001, 256, oracle.PER_ROW, 1.0),
    (40, 257, 128, oracle.MX32, 1.0)])
def test_divergence_matches_oracle(T, V, d, scaling, tau):
    H, W, hq, hs, wq, ws, ids = _case(T, V, d, scaling, T + V)
    got = _gpu(H, W, hq, hs, wq, ws, scaling, ids, tau)
    ref = oracle.divergence(H, W, hq, hs, wq, ws, scaling, inv_temperature=1.0 / tau)
    _check(got, ref, d, _norms(H, W, hq, hs, wq, ws, scaling, tau, range(T)))
    assert np.all(got["kl_pi_mu"] > 0) and np.all(got["l2"] > 0)


def test_passes_masks_and_slots():
    T, V, d, sc = 700, 1000, 256, oracle.PER_ROW
    H, W, hq, hs, wq, ws, ids = _case(T, V, d, sc, 3)
    one = _gpu(H, W, hq, hs, wq, ws, sc, ids, 1.0)
    # passes of 256 rows give the same values
    three = _gpu(H, W, hq, hs, wq, ws, sc, ids, 1.0, div_chunk=256)
    for k in ("kl_pi_mu", "kl_mu_pi", "l2", "logp_pi", "logp_mu", "entropy_pi"):
        assert np.array_equal(one[k], three[k]), k
    # masked rows write 0, rows go to their slots
    torch, dev = torch_dev()
    mask = (np.arange(T) % 5 != 2).astype(np.uint8)
    n_slots = T + 40
    slots = np.random.default_rng(4).permutation(n_slots)[:T].astype(np.int32)
    got = _gpu(H, W, hq, hs, wq, ws, sc, ids, 1.0, mask=up(torch, dev, mask), out_slot=up(torch, dev, slots),
               n_slots=n_slots)
    for k in ("kl_pi_mu", "kl_mu_pi", "l2"):
        assert np.array_equal(got[k][slots][mask == 1], one[k][mask == 1]), k
        assert np.all(got[k][slots][mask == 0] == 0), k
    # the scoring outputs are those of a call without the measures
    plain = _gpu_plain(H, W, hq, hs, wq, ws, sc, ids)
    for k in ("logp_pi", "logp_mu", "entropy_pi", "entropy_mu"):
        np.testing.assert_allclose(one[k], plain[k], rtol=0, atol=2e-6)


def _gpu_plain(H, W, hq, hs, wq, ws, scaling, ids):
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    out = acrl.acrl_score_pi_mu(up_bf16(torch, dev, H), up_bf16(torch, dev, W), up(torch, dev, hq),
                                up(torch, dev, hs), up(torch, dev, wq), up(torch, dev, ws), scaling,
                                up(torch, dev, ids))
    torch.cuda.synchronize()
    return {k: down(v) for k, v in out.items()}


def test_lossless_operands_give_zero():
    # bf16 and e4m3 hold the operands exactly (scales 1): identical logits,
    # identical distributions, every measure exactly 0
    h, w, _ = lossless_integer_case(300, 700, 128, 5)
    for sc in (oracle.PER_TENSOR, oracle.PER_ROW):
        hq, hs = oracle.quantize_fp8(h, sc)
        wq, ws = oracle.quantize_fp8(w, sc)
        ids = np.zeros(300, np.int32)
        got = _gpu(h, w, hq, hs, wq, ws, sc, ids, 1e3)
        for k in ("kl_pi_mu", "kl_mu_pi", "l2"):
            assert np.all(got[k] == 0), (sc, k)


def test_full_size_sampled_rows():
    """d = 4096, V = 151936 (the q8b head), 16384 + 300 rows: two passes of
    33 token tiles (passes of at most 16384 rows share the 66 tiles evenly).
    32 rows against the oracle -- both ends of the call, of each pass, of a
    256-row tile and of a 2048-row block of tiles, one row in every other
    block, the rest seeded at random -- and every row against Pinsker's
    bound."""
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    w = inputs.WORKLOADS["q8b"]
    T = 16384 + 300
    Hd = inputs.hidden_bf16_torch(w, T, dev)
    Wd = inputs.weights_bf16_torch(w, dev)
    hq, hs = acrl.acrl_quantize_fp8(Hd, w.scaling)
    wq, ws = acrl.acrl_quantize_fp8(Wd, w.scaling)
    ids = torch.zeros(T, dtype=torch.int32, device=dev)
    out = acrl.acrl_score_pi_mu(Hd, Wd, hq, hs, wq, ws, w.scaling, ids, divergence=True)
    torch.cuda.synchronize()
    got = {k: down(v) for k, v in out.items()}
    cut = 33 * 256
    edges = [0, 255, 256, 2047, 2048, cut - 1, cut, cut + 1, 16383, 16384, T - 1]
    blocks = [b * 2048 + 1000 for b in range(1, 8)]
    rest = np.random.default_rng(31).choice(T, 32 - len(edges) - len(blocks), replace=False)
    rows = np.unique(np.concatenate([edges, blocks, rest]))
    idx = torch.from_numpy(rows).to(dev)
    Hs = down(Hd[idx].view(torch.int16)).view(np.uint16)
    # the oracle's own quantization of the sampled rows is the GPU's (bit-exact, tested elsewhere);
    # per-tensor scales come from the whole H, so the oracle takes that scale
    hq_o, hs_o = oracle.quantize_fp8(down(Hd.view(torch.int16)).view(np.uint16), w.scaling)
    Wh = down(Wd.view(torch.int16)).view(np.uint16)
    wq_o, ws_o = oracle.quantize_fp8(Wh, w.scaling)
    ref = oracle.divergence(Hs, Wh, hq_o[rows], hs_o, wq_o, ws_o, w.scaling)
    _check(got, ref, w.d, _norms(Hs, Wh, hq_o[rows], hs_o, wq_o, ws_o, w.scaling, 1.0, range(len(rows))), rows)
    assert np.all(got["kl_pi_mu"] > 0) and np.all(got["kl_mu_pi"] > 0)
    assert np.all(got["l2"] <= np.sqrt(2 * np.minimum(got["kl_pi_mu"], got["kl_mu_pi"])) * (1 + 1e-3) + 1e-6)


@pytest.mark.parametrize("name", ["q17b", "mx"])
def test_full_size_other_heads(name):
    """The 1.7B-shaped head with per-row FP8 (d = 2048) and the MXFP8 head
    (d = 5120, tau = 0.7) at V = 151936: 4096 + 300 rows in passes of at
    most 2048 rows (three passes of 6 token tiles), 24 rows against the
    oracle -- both ends of the call and of each pass, a tile edge, the rest
    seeded at random."""
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    w = inputs.WORKLOADS[name]
    tau = 1.0 / w.inv_temperature
    T = 4096 + 300
    Hd = inputs.hidden_bf16_torch(w, T, dev)
    Wd = inputs.weights_bf16_torch(w, dev)
    hq, hs = acrl.acrl_quantize_fp8(Hd, w.scaling)
    wq, ws = acrl.acrl_quantize_fp8(Wd, w.scaling)
    ids = torch.zeros(T, dtype=torch.int32, device=dev)
    out = acrl.acrl_score_pi_mu(Hd, Wd, hq, hs, wq, ws, w.scaling, ids, inv_temperature=w.inv_temperature,
                                divergence=True, div_chunk=2048)
    torch.cuda.synchronize()
    got = {k: down(v) for k, v in out.items()}
    cut = 6 * 256
    edges = [0, 255, 256, cut - 1, cut, 2 * cut - 1, 2 * cut, T - 1]
    rest = np.random.default_rng(37).choice(T, 24 - len(edges), replace=False)
    rows = np.unique(np.concatenate([edges, rest]))
    idx = torch.from_numpy(rows).to(dev)
    Hs = down(Hd[idx].view(torch.int16)).view(np.uint16)
    # the oracle's own quantization of the sampled rows (per-row and MX scales are per row)
    hq_o, hs_o = oracle.quantize_fp8(Hs, w.scaling)
    Wh = down(Wd.view(torch.int16)).view(np.uint16)
    wq_o, ws_o = oracle.quantize_fp8(Wh, w.scaling)
    ref = oracle.divergence(Hs, Wh, hq_o, hs_o, wq_o, ws_o, w.scaling, inv_temperature=w.inv_temperature)
    _check(got, ref, w.d, _norms(Hs, Wh, hq_o, hs_o, wq_o, ws_o, w.scaling, tau, range(len(rows))), rows, tau=tau)
    assert np.all(got["kl_pi_mu"] > 0) and np.all(got["kl_mu_pi"] > 0)


def _scaled_mu_case(T, V, d, scaling, seed, scale, pi_scale=1.0):
    """pi's head pi_scale * W and a mu built from scale * W: the two lse differ
    by several nats (the kernels form the measures relative to mu's lse)."""
    H = random_bf16((T, d), seed)
    W = random_bf16((V, d), seed + 1, std=2.5 / math.sqrt(d))
    Wf = (W.astype(np.uint32) << 16).view(np.float32)
    Wp = inputs.float_to_bf16_bits(Wf * np.float32(pi_scale))
    Wm = inputs.float_to_bf16_bits(Wf * np.float32(scale))
    hq, hs = oracle.quantize_fp8(H, scaling)
    wq, ws = oracle.quantize_fp8(Wm, scaling)
    return H, Wp, hq, hs, wq, ws


def _lse_gap(H, W, hq, hs, wq, ws, scaling, rows):
    """lse_pi - lse_mu of the rows, from the oracle's logits."""
    from scipy.special import logsumexp
    return np.array([logsumexp(oracle.logits_pi(H[r], W, 1.0)) -
                     logsumexp(oracle.logits_mu(hq[r], oracle._row_scale(hs, scaling, r), wq, ws, scaling, 1.0))
                     for r in rows])


@pytest.mark.parametrize("scale", [1.6, 0.9])
def test_distant_policies_match_oracle(scale):
    # mu sharper (lse_pi - lse_mu of -3 to -6 nats) or a little flatter
    # (+0.4 to +0.9): the terms pt = exp(z - lse_mu) are far from p, and the
    # identities still give the oracle's values
    T, V, d, sc = 160, 1000, 256, oracle.PER_ROW
    H, W, hq, hs, wq, ws = _scaled_mu_case(T, V, d, sc, 21, scale)
    ids = np.zeros(T, np.int32)
    got = _gpu(H, W, hq, hs, wq, ws, sc, ids, 1.0)
    ref = oracle.divergence(H, W, hq, hs, wq, ws, sc)
    gap = _lse_gap(H, W, hq, hs, wq, ws, sc, range(T))
    assert (gap.max() < -2.0) if scale > 1 else (0.2 < gap.min() and gap.max() < 2.0), gap
    norms = _norms(H, W, hq, hs, wq, ws, sc, 1.0, range(T))
    _check(got, ref, d, norms)


def test_mu_logit_far_above_pi_at_one_entry():
    # A constant input feature gives pi a large logit at entry 900 (+56) and
    # mu one at entry 5 (+72): |lse_pi - lse_mu| of 5 to 26 nats, so the
    # measures are defined, while at entry 5 mu's logit lies more than 44
    # nats above every pi logit of its vocabulary tile (pi's terms there are
    # ~2^-100 of mu's, and terms formed relative to pi's own running maximum
    # would overflow fp32).  The values match the oracle.
    T, V, d, sc = 64, 1000, 256, oracle.PER_ROW
    H = random_bf16((T, d), 41)
    W = random_bf16((V, d), 42, std=2.5 / math.sqrt(d))
    H[:, 0] = inputs.float_to_bf16_bits(np.ones(T, np.float32))
    Wp, Wm = W.copy(), W.copy()
    Wp[:, 0] = 0
    Wm[:, 0] = 0
    Wp[900, 0] = inputs.float_to_bf16_bits(np.array([56.0], np.float32))[0]
    Wm[5, 0] = inputs.float_to_bf16_bits(np.array([72.0], np.float32))[0]
    hq, hs = oracle.quantize_fp8(H, sc)
    wq, ws = oracle.quantize_fp8(Wm, sc)
    gap = _lse_gap(H, Wp, hq, hs, wq, ws, sc, range(T))
    assert np.all(np.abs(gap) < 32) and np.all(np.abs(gap) > 3), gap
    from scipy.special import logsumexp
    lse = np.zeros((2, T))
    for r in range(T):
        zp = oracle.logits_pi(H[r], Wp, 1.0)
        zm = oracle.logits_mu(hq[r], oracle._row_scale(hs, sc, r), wq, ws, sc, 1.0)
        assert zm[5] - zp[:256].max() > 45
        lse[:, r] = logsumexp(zp), logsumexp(zm)
    got = _gpu(H, Wp, hq, hs, wq, ws, sc, np.zeros(T, np.int32), 1.0)
    ref = oracle.divergence(H, Wp, hq, hs, wq, ws, sc)
    for k in ("kl_pi_mu", "kl_mu_pi", "l2"):
        assert np.all(np.isfinite(got[k])), k
    # Logits near 60-70 carry the matrix cores' accumulation error at their
    # own scale (mu's lse is off by up to ~1e-2 here, against ~1e-4 at the
    # O(1) logits the bound above assumes); each KL moves by at most the two
    # lse errors plus the error of the logits that hold the mass, which the
    # usual bound covers.
    dA = np.abs(got["lse_pi"] - lse[0]) + np.abs(got["lse_mu"] - lse[1])
    np_, nq = _norms(H, Wp, hq, hs, wq, ws, sc, 1.0, range(T))
    delta = 2e-4 * math.sqrt(d / 256.0)
    for k in ("kl_pi_mu", "kl_mu_pi"):
        tol = 1e-6 + 2 * delta * np.sqrt(2 * np.abs(ref[k])) + 2 * dA
        assert np.all(np.abs(got[k] - ref[k]) <= tol), (k, np.abs(got[k] - ref[k]).max())
    assert np.all(np.abs(got["l2"] - ref["l2"]) <= 1e-6 + 2 * delta * (np_ + nq))


def test_far_apart_policies_give_nan():
    # |lse_pi - lse_mu| > 32: every measure is NaN (masked rows still 0)
    T, V, d, sc = 64, 1000, 256, oracle.PER_ROW
    torch, dev = torch_dev()
    mask = (np.arange(T) % 4 != 1).astype(np.uint8)
    H, W, hq, hs, wq, ws = _scaled_mu_case(T, V, d, sc, 23, 25.0)
    assert _lse_gap(H, W, hq, hs, wq, ws, sc, range(T)).max() < -32
    got = _gpu(H, W, hq, hs, wq, ws, sc, np.zeros(T, np.int32), 1.0, mask=up(torch, dev, mask))
    for k in ("kl_pi_mu", "kl_mu_pi", "l2"):
        assert np.all(np.isnan(got[k][mask == 1])), k
        assert np.all(got[k][mask == 0] == 0), k
    # pi's lse 5 to 8 nats above mu's: the three terms of the distance cancel
    # beyond fp32's reach, so it is NaN; both KL stay finite and match
    H, W, hq, hs, wq, ws = _scaled_mu_case(T, V, d, sc, 25, 0.2, pi_scale=1.6)
    gap = _lse_gap(H, W, hq, hs, wq, ws, sc, range(T))
    assert gap.min() > 4 and gap.max() < 32, gap
    got = _gpu(H, W, hq, hs, wq, ws, sc, np.zeros(T, np.int32), 1.0)
    ref = oracle.divergence(H, W, hq, hs, wq, ws, sc)
    assert np.all(np.isnan(got["l2"]))
    delta = 2e-4 * math.sqrt(d / 256.0)
    for k in ("kl_pi_mu", "kl_mu_pi"):
        tol = 1e-6 + 2 * delta * np.sqrt(2 * np.abs(ref[k])) + 1e-5 * np.abs(ref[k])
        assert np.all(np.abs(got[k] - ref[k]) <= tol), (k, np.abs(got[k] - ref[k]).max())
