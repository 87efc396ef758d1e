"""Shared test cases: seeded inputs (from inputs/) plus oracle-derived fixtures.

Token ids of the small workload are sampled from the oracle's mu (inverse
CDF with seeded uniforms), as the workload prescribes; nothing here comes from
the HIP path.  Tolerances are the acceptance bounds of the scoring path.
"""
import math

import numpy as np

import inputs
import oracle

# acceptance bounds (per token / per sequence)
TOL_LOGP = 2e-3                      # |logp_gpu - logp_oracle|


def tol_entropy(V: int) -> float:    # |H_gpu - H_oracle|
    return 1e-3 * math.log(V)


def tol_seq_logratio(n: int) -> float:  # |sum_t log(pi/mu)| per sequence
    return 1e-3 * math.sqrt(max(n, 1))


def oracle_sampled_ids(H, hq, hs, wq, ws, scaling, inv_temperature, u):
    """Ids drawn from the oracle's mu for every row of H."""
    z = np.stack([oracle.logits_mu(hq[r], oracle._row_scale(hs, scaling, r), wq, ws, scaling,
                                   inv_temperature) for r in range(H.shape[0])])
    return oracle.sample_inverse_cdf(z, u)


def workload_case(name: str):
    """The whole small workload: valid rows packed sequence-major."""
    w = inputs.WORKLOADS[name]
    n = inputs.n_valid(w)
    H = inputs.hidden_bf16(w)
    W = inputs.weights_bf16(w)
    hq, hs = oracle.quantize_fp8(H, w.scaling)
    wq, ws = oracle.quantize_fp8(W, w.scaling)
    ids = oracle_sampled_ids(H, hq, hs, wq, ws, w.scaling, w.inv_temperature, inputs.uniforms(w, n))
    return dict(w=w, H=H, W=W, hq=hq, hs=hs, wq=wq, ws=ws, ids=ids,
                slots=inputs.valid_slots(w), mask=inputs.mask(w), groups=inputs.group_of_seq(w),
                adv=inputs.advantages(w))


def random_bf16(shape, seed, std=1.0):
    r = np.random.default_rng(seed)
    return inputs.float_to_bf16_bits((r.standard_normal(shape) * std).astype(np.float32))


def lossless_integer_case(T, V, d, seed):
    """Integer operands that are exact in bf16 and e4m3 with every FP8 scale
    equal to 1 (each row of H and of W holds a 448 in a column where the other
    operand is zero), so pi and mu logits are the same exact integers."""
    assert d >= 8
    r = np.random.default_rng(seed)
    h = r.integers(-4, 5, size=(T, d)).astype(np.float32)
    w = r.integers(-4, 5, size=(V, d)).astype(np.float32)
    h[:, 0], w[:, 0] = 448.0, 0.0
    h[:, 1], w[:, 1] = 0.0, 448.0
    z = (w.astype(np.int64) @ h.astype(np.int64).T).T  # [T, V] exact
    return inputs.float_to_bf16_bits(h), inputs.float_to_bf16_bits(w), z
