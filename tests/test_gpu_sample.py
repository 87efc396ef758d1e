"""GPU parity of acrl_sample_mu (blockwise Gumbel-max draw from mu, fused
into the mu kernel) with the oracle's blockwise sampler on the same
counter-based uniforms (Philox4x32-10).

The draw has two steps.  First a block of 16 vocabulary rows wins by
Gumbel-max over the blocks' keys.  Then the row inside it comes from the
inverse CDF of the block's softmax.  Floating point decides both steps.
The kernel uses fp32 logits and the hardware log2; the oracle uses fp64.
The kernel's block must have a key within rounding of the oracle's best
key; where the oracle's best block clears the runner-up by more than
that, the blocks must match.  The row must be the oracle's pick in that
block, unless u' falls within rounding of a cumulative-probability
boundary; then it must be a row whose interval touches u'.  The sampled
log-prob is checked like the scorer's (2e-3)."""
import numpy as np
import pytest

import inputs
import oracle
from cases import TOL_LOGP, random_bf16
from gpu_util import down, par_map, torch_dev, up, up_bf16

pytestmark = pytest.mark.gpu

KEY_TOL = 2e-3  # fp32 logits (~1e-5 relative) and the hardware log2 against fp64
CUM_TOL = 1e-4  # fp32 exponentials and running sums of 16 weights


def _check_draw(z, ids, seed, row_offset, tokens=None, key_tol=KEY_TOL):
    n, V = z.shape
    n_clear = 0
    for r in range(n):
        t = row_offset + r if tokens is None else int(tokens[r])
        keys = oracle.block_gumbel_keys(z[r], seed, t)
        best = keys.max()
        kg = int(oracle.block_of_row(ids[r]))
        assert keys[kg] >= best - key_tol, (r, keys[kg], best)
        srt = np.sort(keys)
        if srt[-1] - srt[-2] > key_tol:
            n_clear += 1
            assert kg == int(np.argmax(keys)), r
        row, cum, u = oracle.block_pick(z[r], seed, t, kg)
        if ids[r] != row:
            slots = oracle.block_slot_rows(kg, V)
            q = int(np.flatnonzero(slots == ids[r])[0])
            lo = 0.0 if q == 0 else np.nanmax(np.concatenate([[0.0], cum[:q]]))
            assert lo - CUM_TOL <= u <= cum[q] + CUM_TOL, (r, lo, u, cum[q])
    return n_clear


@pytest.mark.parametrize("scaling", [oracle.PER_ROW, oracle.PER_TENSOR, oracle.MX32])
@pytest.mark.parametrize("T,V,d,inv_temp", [(300, 1000, 256, 1.0), (65, 300, 128, 1 / 0.7), (40, 2048, 128, 1.0)])
def test_sample_matches_oracle(scaling, T, V, d, inv_temp):
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    H = random_bf16((T, d), 41 + T)
    W = random_bf16((V, d), 42 + V, std=2.5 / np.sqrt(d))
    h, w = up_bf16(torch, dev, H), up_bf16(torch, dev, W)
    hq, hs = acrl.acrl_quantize_fp8(h, scaling)
    wq, ws = acrl.acrl_quantize_fp8(w, scaling)
    seed, off = 0x1234_5678_9ABC, 1000
    ids, lp = acrl.acrl_sample_mu(hq, hs, wq, ws, scaling, seed, row_offset=off, inv_temperature=inv_temp)
    torch.cuda.synchronize()
    ids, lp = down(ids), down(lp)
    assert ((ids >= 0) & (ids < V)).all()
    # the oracle's own quantization (bit-exact with the device's, checked here too)
    hq_o, hs_o = oracle.quantize_fp8(H, scaling)
    wq_o, ws_o = oracle.quantize_fp8(W, scaling)
    assert np.array_equal(down(hq), hq_o) and np.array_equal(down(wq), wq_o)
    z = np.stack([oracle.logits_mu(hq_o[r], oracle._row_scale(hs_o, scaling, r), wq_o, ws_o, scaling, inv_temp)
                  for r in range(T)])
    n_clear = _check_draw(z, ids, seed, off)
    assert n_clear > 0.9 * T
    want, _, _ = oracle.block_gumbel_sample(z, seed, off)
    assert (ids == want).mean() > 0.95
    # log mu of the drawn row
    lse = np.log(np.exp(z - z.max(axis=1, keepdims=True)).sum(axis=1)) + z.max(axis=1)
    np.testing.assert_allclose(lp, z[np.arange(T), ids] - lse, atol=TOL_LOGP, rtol=0)


@pytest.mark.parametrize("name", ["q8b", "q17b", "mx"])
def test_full_size_heads_sampled_rows(name):
    """The draw at V = 151936 on the workloads' heads (per-tensor FP8 at
    d = 4096, per-row FP8 at d = 2048, MXFP8 at d = 5120 and tau = 0.7) for
    4096 + 300 rows in one call: 24 rows -- both ends of the call and of a
    tile, the rest seeded -- against the oracle's blockwise draw on the same
    counters.  The logits of the FP8 products sit up to ~2e-4 sqrt(d / 256)
    / tau from the oracle's exact ones, so the keys get that much more room."""
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    w = inputs.WORKLOADS[name]
    T = 4096 + 300
    Hd = inputs.hidden_bf16_torch(w, T, dev)
    Wd = inputs.weights_bf16_torch(w, dev)
    hq, hs = acrl.acrl_quantize_fp8(Hd, w.scaling)
    wq, ws = acrl.acrl_quantize_fp8(Wd, w.scaling)
    seed, off = 0x0DDB_A11, 123456
    ids, lp = acrl.acrl_sample_mu(hq, hs, wq, ws, w.scaling, seed, row_offset=off,
                                  inv_temperature=w.inv_temperature)
    torch.cuda.synchronize()
    ids, lp = down(ids), down(lp)
    assert ((ids >= 0) & (ids < w.V)).all()
    edges = [0, 255, 256, T - 1]
    rows = np.unique(np.concatenate([edges, np.random.default_rng(43).choice(T, 24 - len(edges), replace=False)]))
    # the oracle's own quantization: of the whole H for the per-tensor scale, of the rows otherwise
    H = down(Hd.view(torch.int16)).view(np.uint16)
    Wh = down(Wd.view(torch.int16)).view(np.uint16)
    hq_o, hs_o = oracle.quantize_fp8(H if w.scaling == oracle.PER_TENSOR else H[rows], w.scaling)
    if w.scaling == oracle.PER_TENSOR:
        hq_o = hq_o[rows]
    wq_o, ws_o = oracle.quantize_fp8(Wh, w.scaling)
    oracle.lib()
    z = np.stack(par_map(lambda k: oracle.logits_mu(hq_o[k], oracle._row_scale(hs_o, w.scaling, k), wq_o, ws_o,
                                                    w.scaling, w.inv_temperature), range(len(rows))))
    key_tol = KEY_TOL * max(1.0, np.sqrt(w.d / 256.0) * w.inv_temperature)
    n_clear = _check_draw(z, ids[rows], seed, 0, tokens=off + rows, key_tol=key_tol)
    assert n_clear > 0.8 * len(rows)
    want = np.array([oracle.block_gumbel_sample(z[k:k + 1], seed, off + int(r))[0][0] for k, r in enumerate(rows)])
    assert (ids[rows] == want).mean() > 0.9
    lse = np.log(np.exp(z - z.max(axis=1, keepdims=True)).sum(axis=1)) + z.max(axis=1)
    np.testing.assert_allclose(lp[rows], z[np.arange(len(rows)), ids[rows]] - lse, atol=TOL_LOGP, rtol=0)


def test_sample_chunked_equals_one_shot_and_frequencies():
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    T, V, d = 4096, 64, 128
    H = random_bf16((T, d), 5)
    W = random_bf16((V, d), 6, std=0.3)
    # every row the same hidden state: the draws are iid from one softmax
    H[:] = H[0]
    h, w = up_bf16(torch, dev, H), up_bf16(torch, dev, W)
    hq, hs = acrl.acrl_quantize_fp8(h, oracle.PER_ROW)
    wq, ws = acrl.acrl_quantize_fp8(w, oracle.PER_ROW)
    a, _ = acrl.acrl_sample_mu(hq, hs, wq, ws, oracle.PER_ROW, 99)
    b = torch.empty_like(a)
    for r0 in range(0, T, 1000):
        r1 = min(T, r0 + 1000)
        acrl.acrl_sample_mu(hq[r0:r1], hs[r0:r1], wq, ws, oracle.PER_ROW, 99, row_offset=r0, ids=b[r0:r1],
                            want_logp=False)
    torch.cuda.synchronize()
    a, b = down(a), down(b)
    assert np.array_equal(a, b)
    hq_o, hs_o = oracle.quantize_fp8(H[:1], oracle.PER_ROW)
    wq_o, ws_o = oracle.quantize_fp8(W, oracle.PER_ROW)
    z = oracle.logits_mu(hq_o[0], oracle._row_scale(hs_o, oracle.PER_ROW, 0), wq_o, ws_o, oracle.PER_ROW, 1.0)
    p = np.exp(z - z.max())
    p /= p.sum()
    freq = np.bincount(a, minlength=V) / T
    sigma = np.sqrt(p * (1 - p) / T)
    # 5 standard deviations, plus two draws of slack for rows whose expected
    # count is far below one (a single draw of such a row is not a bias)
    assert (np.abs(freq - p) < 5 * sigma + 2.0 / T).all()
