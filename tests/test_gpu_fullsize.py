"""Full-size parity of acrl_score_pi_mu with the oracle, in the launch
configuration the benchmark times: the whole batch of a workload scored in
one call into its [B, L] slots, with the token ids drawn from mu
(acrl_sample_mu, Gumbel-max at the workload's temperature, seed = the
workload's seed), as the rollout tokens of the paper are (a_t ~ mu, Sec. 2).
The ids are inputs to both sides.

Per workload (q8b, q17b, mx, long):
  * at least 256 valid rows, one in every block of 8 token tiles (the 2048
    rows an XCD's block of workgroups covers), the last partial block
    included, and the rest stratified over the batch; the oracle scores each
    at full V and d with its own FP8 quantization;
  * per-token bounds: |logp| <= 2e-3, |entropy| <= 1e-3 log V, lse and the
    gathered logit <= 2e-3;
  * the binding per-sequence bound |sum log(pi/mu) - oracle| <= 1e-3 sqrt(n)
    (rho_i of Eq. mis_objective, built from the probabilities of
    Eq. distance_metric) is checked on the workload's longest response from
    the per-token errors: with e_t = log-ratio error of token t, mean m and
    standard deviation s over the sampled rows, n m + 3 s sqrt(n) must stay
    within 1e-3 sqrt(n) (a systematic per-token bias adds up linearly in n,
    the rest like sqrt(n));
  * whole responses: the shortest q8b response (1024 tokens, d = 4096) and
    the shortest mx response (523 tokens, d = 5120) go through the oracle's
    whole chain (quantization, scores, reduce of that response) and their
    sums of log-ratios are compared with the device's reduce output.

Every check prints the measured errors (mean and spread of the log-ratio
error, of mu's gathered logit and its slope against the logit) so that a
systematic error of the FP8 products is visible in the run's output.
"""
import math

import numpy as np
import pytest

import inputs
import oracle
from cases import TOL_LOGP, tol_entropy, tol_seq_logratio
from gpu_util import down, torch_dev, up

pytestmark = pytest.mark.gpu

MIN_ROWS = 256
BLOCK_ROWS = 8 * 256  # token rows of one 8-token-tile block of workgroups

_state = {}  # one workload's device batch and oracle operands at a time


def _say(*a):
    print(*a, flush=True)


def _release():
    _state.clear()
    import torch
    torch.cuda.empty_cache()


def _batch(name):
    """The workload scored and reduced on the device as the benchmark does."""
    if _state.get("name") == name:
        return _state
    _release()
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    w = inputs.WORKLOADS[name]
    T = inputs.n_valid(w)
    slots = inputs.valid_slots(w)
    h = inputs.hidden_bf16_torch(w, T, dev)
    W = inputs.weights_bf16_torch(w, dev)
    wq, ws = acrl.acrl_quantize_fp8(W, w.scaling)
    hq, hs = acrl.acrl_quantize_fp8(h, w.scaling)
    ids, _ = acrl.acrl_sample_mu(hq, hs, wq, ws, w.scaling, seed=w.seed, inv_temperature=w.inv_temperature,
                                 want_logp=False)
    sc = acrl.acrl_score_pi_mu(h, W, hq, hs, wq, ws, w.scaling, ids, inv_temperature=w.inv_temperature,
                               out_slot=up(torch, dev, slots), n_slots=w.slots)
    mask = inputs.mask(w)
    groups = inputs.group_of_seq(w)
    red = acrl.acrl_discrepancy_reduce(w.B, w.L, w.n_prompts, sc["logp_pi"], sc["logp_mu"],
                                       up(torch, dev, mask.reshape(-1)), up(torch, dev, groups),
                                       entropy_pi=sc["entropy_pi"], entropy_mu=sc["entropy_mu"])
    torch.cuda.synchronize()
    ids_np = down(ids)
    assert ((ids_np >= 0) & (ids_np < w.V)).all()
    _state.update(name=name, w=w, T=T, slots=slots, h=h, ids=ids_np,
                  gpu={k: down(v)[slots] for k, v in sc.items()},
                  red={k: down(v) for k, v in red.items() if v is not None and not k.startswith("_")})
    del W, wq, hq, sc
    # the oracle's own quantization of W, and of the whole of H for the
    # per-tensor scale (the device codes never feed the oracle)
    _state["W_bits"] = inputs.weights_bf16_torch(w, dev).cpu().view(torch.int16).numpy().view(np.uint16)
    _state["wq_o"], _state["ws_o"] = oracle.quantize_fp8(_state["W_bits"], w.scaling)
    if w.scaling == oracle.PER_TENSOR:
        _state["hq_tensor_o"], _state["hs_tensor_o"] = oracle.quantize_fp8(
            h.cpu().view(torch.int16).numpy().view(np.uint16), w.scaling)
    _say("[%s] batch of %d valid tokens scored on the device; oracle W quantized" % (name, T))
    return _state


def _oracle_rows(st, rows):
    """The oracle's scores of the given valid rows (full V, full d)."""
    import torch
    w = st["w"]
    idx = torch.from_numpy(np.ascontiguousarray(rows, np.int64)).to(st["h"].device)
    Hs = st["h"].index_select(0, idx).cpu().view(torch.int16).numpy().view(np.uint16)
    if w.scaling == oracle.PER_TENSOR:
        # the scale belongs to the whole of H: the rows' codes from the
        # oracle's quantization of the whole tensor
        hq_o, hs_o = st["hq_tensor_o"][rows], st["hs_tensor_o"]
    else:
        hq_o, hs_o = oracle.quantize_fp8(Hs, w.scaling)
    return oracle.score(Hs, st["W_bits"], hq_o, hs_o, st["wq_o"], st["ws_o"], w.scaling, st["ids"][rows],
                        inv_temperature=w.inv_temperature)


def _rows_for(T, seed):
    r = np.random.default_rng(seed)
    n_blocks = (T + BLOCK_ROWS - 1) // BLOCK_ROWS
    per_block = [min(b * BLOCK_ROWS + r.integers(0, BLOCK_ROWS), T - 1) for b in range(n_blocks)]
    n_strata = max(MIN_ROWS - n_blocks, 0)
    edges = np.linspace(0, T, n_strata + 1).astype(np.int64)
    strata = [int(r.integers(edges[i], max(edges[i + 1], edges[i] + 1))) for i in range(n_strata)]
    extra = [0, 255, 256, T - 1, (T - 1) // 256 * 256]  # first / last rows, a tile edge, the last tile
    rows = np.unique(np.concatenate([per_block, strata, extra]).astype(np.int64))
    rows = rows[(rows >= 0) & (rows < T)]
    assert rows.size >= MIN_ROWS
    assert set(rows // BLOCK_ROWS) == set(range(n_blocks))  # every block, the partial last one too
    return rows


def _check_tokens(st, rows, ref):
    w = st["w"]
    g = {k: v[rows] for k, v in st["gpu"].items()}
    for tag in ("pi", "mu"):
        dl = np.abs(g["logp_" + tag] - ref["logp_" + tag])
        assert dl.max() <= TOL_LOGP, "logp_%s off by %g" % (tag, dl.max())
        de = np.abs(g["entropy_" + tag] - ref["ent_" + tag])
        assert de.max() <= tol_entropy(w.V), "entropy_%s off by %g" % (tag, de.max())
        ds = np.abs(g["lse_" + tag] - ref["lse_" + tag])
        assert ds.max() <= TOL_LOGP, "lse_%s off by %g" % (tag, ds.max())
        dz = np.abs(g["logit_" + tag] - ref["z_" + tag])
        assert dz.max() <= TOL_LOGP, "logit_%s off by %g" % (tag, dz.max())
    return g


def _report(name, g, ref):
    """Signed errors against the oracle, printed; returns the log-ratio errors."""
    e = (g["logp_pi"].astype(np.float64) - g["logp_mu"]) - (ref["logp_pi"] - ref["logp_mu"])
    out = {"n": e.size, "lr_mean": e.mean(), "lr_std": e.std(ddof=1), "lr_absmax": np.abs(e).max()}
    for tag in ("pi", "mu"):
        dz = g["logit_" + tag].astype(np.float64) - ref["z_" + tag]
        dl = g["lse_" + tag].astype(np.float64) - ref["lse_" + tag]
        dp = g["logp_" + tag].astype(np.float64) - ref["logp_" + tag]
        z = ref["z_" + tag]
        slope = float(np.dot(dz, z) / np.dot(z, z))  # least-squares dz ~ slope * z
        out.update({"logit_%s_mean" % tag: dz.mean(), "logit_%s_std" % tag: dz.std(ddof=1),
                    "logit_%s_slope" % tag: slope, "lse_%s_mean" % tag: dl.mean(),
                    "logp_%s_mean" % tag: dp.mean(), "logp_%s_std" % tag: dp.std(ddof=1)})
    _say("[%s] errors vs oracle: " % name + ", ".join("%s=%.3g" % (k, v) for k, v in out.items()))
    return e


def _rows_case(name):
    st = _batch(name)
    w, T = st["w"], st["T"]
    rows = _rows_for(T, w.seed + 1000)
    ref = _oracle_rows(st, rows)
    g = _check_tokens(st, rows, ref)
    e = _report(name, g, ref)
    # the binding bound on the workload's longest response
    n_max = int(inputs.lengths(w).max())
    m, s = float(e.mean()), float(e.std(ddof=1))
    worst = n_max * abs(m) + 3 * s * math.sqrt(n_max)
    _say("[%s] longest response n=%d: n|mean| + 3 std sqrt(n) = %.4g, bound %.4g"
         % (name, n_max, worst, tol_seq_logratio(n_max)))
    assert worst <= tol_seq_logratio(n_max)
    # every slot's outputs are finite and in range
    lp = st["gpu"]["logp_pi"]
    ent = st["gpu"]["entropy_pi"]
    assert np.isfinite(lp).all() and (lp <= 1e-6).all()
    assert (ent >= -1e-4).all() and (ent <= math.log(w.V) + 1e-3).all()
    assert np.isfinite(st["gpu"]["logp_mu"]).all()


# the shortest q8b response is scored by the oracle in two halves (two tests,
# so that no single test runs the oracle for much more than a minute); the
# last part of a workload checks the response's sum
_SEQ_PARTS = {"q8b": 2, "mx": 1}
_seq_done = {}


def _response_case(name, part):
    st = _batch(name)
    w = st["w"]
    n = inputs.lengths(w)
    i = int(np.argmin(n))
    seq_rows = np.flatnonzero(st["slots"] // w.L == i)
    assert seq_rows.size == n[i]
    parts = _SEQ_PARTS[name]
    lo, hi = part * seq_rows.size // parts, (part + 1) * seq_rows.size // parts
    ref = _oracle_rows(st, seq_rows[lo:hi])
    _check_tokens(st, seq_rows[lo:hi], ref)
    _seq_done[(name, part)] = ref
    _say("[%s] response %d (%d tokens): part %d of %d scored by the oracle" % (name, i, n[i], part + 1, parts))
    if part + 1 < parts:
        return
    missing = [p for p in range(parts) if (name, p) not in _seq_done]
    assert not missing, "parts %s of the response were not scored" % missing
    cat = {k: np.concatenate([_seq_done[(name, p)][k] for p in range(parts)]) for k in ("logp_pi", "logp_mu")}
    # the oracle's reduce over a batch holding just this response
    lp_pi = np.zeros(w.L)
    lp_mu = np.zeros(w.L)
    lp_pi[: n[i]] = cat["logp_pi"]
    lp_mu[: n[i]] = cat["logp_mu"]
    m1 = (np.arange(w.L) < n[i]).astype(np.uint8)[None, :]
    oref = oracle.discrepancy_reduce(1, w.L, lp_pi, lp_mu, m1, np.zeros(1, np.int32), 1)
    assert st["red"]["seq_len"][i] == oref["seq_len"][0] == n[i]
    got = float(st["red"]["seq_sum_logratio"][i])
    want = float(oref["seq_sum_logratio"][0])
    _say("[%s] response %d: sum log(pi/mu) device %.6g, oracle %.6g, difference %.3g, bound %.3g"
         % (name, i, got, want, got - want, tol_seq_logratio(n[i])))
    assert abs(got - want) <= tol_seq_logratio(n[i])
    # the sum of d = |pi - mu| moves by at most about p |dlogp| per token
    pmax = np.maximum(np.exp(lp_pi), np.exp(lp_mu))
    assert abs(st["red"]["seq_sum_d"][i] - oref["seq_sum_d"][0]) <= 2 * 2 * TOL_LOGP * pmax.sum() + 1e-12


# each workload's cases run back to back (its device batch and oracle
# operands are built once)
@pytest.mark.parametrize("case", ["q8b-rows", "q8b-response-0", "q8b-response-1", "mx-rows", "mx-response-0",
                                  "q17b-rows", "long-rows"])
def test_fullsize_mu_drawn_ids(case):
    parts = case.split("-")
    if parts[1] == "rows":
        _rows_case(parts[0])
    else:
        _response_case(parts[0], int(parts[2]))


def test_zz_release_fullsize():
    # frees the last workload's device buffers before the files after this one
    _release()
