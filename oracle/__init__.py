"""CPU oracle for the ACRL scoring / discrepancy path -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its binding) never imports, links or runs it.

The oracle is the plain C file ``acrl_oracle.c`` (fp64, written from the ACRL
paper's definitions, independent of the HIP sources).  This module builds it
with gcc and exposes numpy-level wrappers.  Function-level citations live in
the C source.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "acrl_oracle.c")
LIB = os.path.join(HERE, "libacrl_oracle.so")

PER_TENSOR, PER_ROW, MX32 = 0, 1, 2
ROUND_NEAREST_EVEN, ROUND_TOWARD_ZERO = 0, 1
Y_GROUP, Y_SEQUENCE, Y_BATCH = 0, 1, 2
CTRL_ACRL, CTRL_TIS, CTRL_MIS, CTRL_CONTINUOUS, CTRL_FALLBACK = 0, 1, 2, 3, 4

# indices of the batch statistics vector (mirrors the enum in acrl_oracle.h)
STAT_Y_BATCH = 0
STAT_TOK_MEAN_D = 1
STAT_TOK_MAX_D = 2
STAT_TOK_STD_D = 3
STAT_MEAN_H_PI = 4
STAT_MEAN_H_MU = 5
STAT_N_TOKENS = 6
STAT_N_GROUPS = 7
STAT_TOK_MEAN_LOGRATIO = 8
STAT_N_SEQS = 9
N_STATS = 10


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no fast-math, OpenMP across tokens)."""
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        tmp = LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
               "-fno-fast-math", "-ffp-contract=off", "-Wall", "-Wextra",
               "-o", tmp, SRC, "-lm"]
        subprocess.run(cmd, check=True, cwd=HERE)
        os.replace(tmp, LIB)
    return LIB


_lib: Optional[ctypes.CDLL] = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build(force=False)
        L = ctypes.CDLL(LIB)
        P, I64, I32, D = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_double
        L.acrl_ref_bf16_to_float.restype = ctypes.c_float
        L.acrl_ref_bf16_to_float.argtypes = [ctypes.c_uint16]
        L.acrl_ref_e4m3_encode.restype = ctypes.c_uint8
        L.acrl_ref_e4m3_encode.argtypes = [ctypes.c_float, I32]
        L.acrl_ref_e4m3_decode.restype = D
        L.acrl_ref_e4m3_decode.argtypes = [ctypes.c_uint8]
        L.acrl_ref_e8m0_decode.restype = D
        L.acrl_ref_e8m0_decode.argtypes = [ctypes.c_uint8]
        L.acrl_ref_e4m3_encode_array.restype = None
        L.acrl_ref_e4m3_encode_array.argtypes = [P, I64, I32, P]
        L.acrl_ref_quantize_fp8.restype = I32
        L.acrl_ref_quantize_fp8.argtypes = [P, I64, I64, I64, I32, I32, P, P]
        L.acrl_ref_logits_pi.restype = I32
        L.acrl_ref_logits_pi.argtypes = [P, P, I64, I64, D, P]
        L.acrl_ref_logits_mu.restype = I32
        L.acrl_ref_logits_mu.argtypes = [P, P, P, P, I32, I64, I64, D, P]
        L.acrl_ref_token_stats.restype = None
        L.acrl_ref_token_stats.argtypes = [P, I64, ctypes.c_int32, P, P, P]
        L.acrl_ref_score.restype = I32
        L.acrl_ref_score.argtypes = [I64, I64, I64, P, P, P, P, P, P, I32, P, P, D] + [P] * 8
        L.acrl_ref_token_divergence.restype = None
        L.acrl_ref_token_divergence.argtypes = [P, P, I64, P, P, P]
        L.acrl_ref_divergence.restype = I32
        L.acrl_ref_divergence.argtypes = [I64, I64, I64, P, P, P, P, P, P, I32, P, D, P, P, P]
        L.acrl_ref_discrepancy_reduce.restype = I32
        L.acrl_ref_discrepancy_reduce.argtypes = [I64, I64, P, P, P, P, P, P, I64] + [P] * 8
        L.acrl_ref_controller_step.restype = I32
        L.acrl_ref_controller_step.argtypes = [I64, I64, P, P, I64, P, P, P, I32, I32, P, P, P,
                                               D, D, D, I32, D, P, P]
        L.acrl_ref_philox4x32_10.restype = None
        L.acrl_ref_philox4x32_10.argtypes = [P, P, P]
        L.acrl_ref_sample_uniform.restype = D
        L.acrl_ref_sample_uniform.argtypes = [ctypes.c_uint64, I64, I64]
        L.acrl_ref_block_gumbel_sample.restype = I32
        L.acrl_ref_block_gumbel_sample.argtypes = [P, I64, I64, ctypes.c_uint64, I64, P, P, P]
        L.acrl_ref_block_gumbel_keys.restype = I32
        L.acrl_ref_block_gumbel_keys.argtypes = [P, I64, ctypes.c_uint64, I64, P]
        L.acrl_ref_block_pick.restype = I64
        L.acrl_ref_block_pick.argtypes = [P, I64, ctypes.c_uint64, I64, I64, P, P]
        L.acrl_ref_gumbel_sample.restype = I32
        L.acrl_ref_gumbel_sample.argtypes = [P, I64, I64, ctypes.c_uint64, I64, P, P]
        L.acrl_ref_reference_x.restype = I32
        L.acrl_ref_reference_x.argtypes = [P, P, I64, P]
        L.acrl_ref_sample_inverse_cdf.restype = I32
        L.acrl_ref_sample_inverse_cdf.argtypes = [P, I64, I64, P, P]
        L.acrl_ref_surrogate.restype = I32
        L.acrl_ref_surrogate.argtypes = [I64, I64, P, P, I64, P, P, P, I32, P, D, D, P, P]
        L.acrl_ref_lm_head_backward.restype = I32
        L.acrl_ref_lm_head_backward.argtypes = [I64, I64, I64, P, P, P, P, D, I64, P, P, P, I64, P, P, P]
        _lib = L
    return _lib


def set_threads(n: int) -> None:
    """Number of OpenMP threads the oracle's loops use from the calling thread
    on (for timing it; the results do not depend on it)."""
    lib()
    ctypes.CDLL("libgomp.so.1").omp_set_num_threads(int(n))


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _check(rc: int, what: str) -> None:
    if rc != 0:
        raise ValueError("oracle %s rejected its arguments" % what)


# ---------------------------------------------------------------- formats
def bf16_to_float(bits: np.ndarray) -> np.ndarray:
    """Exact value of bf16 bit patterns (uint16) as float32."""
    b = _c(bits, np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def e4m3_encode(x, rounding: int = ROUND_NEAREST_EVEN) -> np.ndarray:
    x = _c(x, np.float32)
    out = np.empty(x.shape, np.uint8)
    lib().acrl_ref_e4m3_encode_array(_p(x), x.size, rounding, _p(out))
    return out


def e4m3_decode(codes) -> np.ndarray:
    codes = _c(codes, np.uint8)
    f = lib().acrl_ref_e4m3_decode
    return np.array([f(int(c)) for c in codes.ravel()], np.float64).reshape(codes.shape)


def e8m0_decode(codes) -> np.ndarray:
    codes = _c(codes, np.uint8)
    f = lib().acrl_ref_e8m0_decode
    return np.array([f(int(c)) for c in codes.ravel()], np.float64).reshape(codes.shape)


# ---------------------------------------------------------------- a1/a2
def quantize_fp8(x_bf16: np.ndarray, scaling: int, rounding: int = ROUND_NEAREST_EVEN):
    """x_bf16: uint16 [rows, cols].  Returns (codes uint8 [rows, cols], scales)."""
    x = _c(x_bf16, np.uint16)
    rows, cols = x.shape
    q = np.empty((rows, cols), np.uint8)
    if scaling == PER_TENSOR:
        s = np.empty(1, np.float32)
    elif scaling == PER_ROW:
        s = np.empty(rows, np.float32)
    else:
        s = np.empty((rows, max(cols // 32, 0)), np.uint8)
    _check(lib().acrl_ref_quantize_fp8(_p(x), rows, cols, cols, scaling, rounding, _p(q), _p(s)),
           "quantize")
    return q, s


# ---------------------------------------------------------------- a3/a4
def logits_pi(h_row: np.ndarray, w: np.ndarray, inv_temperature: float = 1.0) -> np.ndarray:
    h_row, w = _c(h_row, np.uint16), _c(w, np.uint16)
    V, d = w.shape
    z = np.empty(V, np.float64)
    _check(lib().acrl_ref_logits_pi(_p(h_row), _p(w), d, V, inv_temperature, _p(z)), "logits_pi")
    return z


def _row_scale(hq_scales: np.ndarray, scaling: int, r: int) -> np.ndarray:
    if scaling == PER_TENSOR:
        return _c(hq_scales.reshape(-1)[:1], np.float32)
    if scaling == PER_ROW:
        return _c(hq_scales.reshape(-1)[r:r + 1], np.float32)
    return _c(hq_scales[r], np.uint8)


def logits_mu(hq_row, row_scale, wq, wq_scales, scaling: int,
              inv_temperature: float = 1.0) -> np.ndarray:
    hq_row, wq = _c(hq_row, np.uint8), _c(wq, np.uint8)
    V, d = wq.shape
    rs = _c(row_scale, np.uint8 if scaling == MX32 else np.float32)
    ws = _c(wq_scales, np.uint8 if scaling == MX32 else np.float32)
    z = np.empty(V, np.float64)
    _check(lib().acrl_ref_logits_mu(_p(hq_row), _p(rs), _p(wq), _p(ws), scaling, d, V,
                                    inv_temperature, _p(z)), "logits_mu")
    return z


def token_stats(z: np.ndarray, token_id: int):
    """(lse, logp, entropy) of one token's logits."""
    z = _c(z, np.float64)
    out = np.zeros(3, np.float64)
    L = lib()
    L.acrl_ref_token_stats(_p(z), z.size, int(token_id), _p(out[0:1]), _p(out[1:2]), _p(out[2:3]))
    return float(out[0]), float(out[1]), float(out[2])


def score(h, w, hq, hq_scales, wq, wq_scales, scaling: int, ids, mask=None,
          inv_temperature: float = 1.0) -> dict:
    """Both policies for every row of h.  Returns a dict of float64 [n_rows]."""
    h, w = _c(h, np.uint16), _c(w, np.uint16)
    hq, wq = _c(hq, np.uint8), _c(wq, np.uint8)
    n_rows, d = h.shape
    V = w.shape[0]
    sdt = np.uint8 if scaling == MX32 else np.float32
    hs, ws = _c(hq_scales, sdt), _c(wq_scales, sdt)
    ids = _c(ids, np.int32)
    m = None if mask is None else _c(mask, np.uint8)
    names = ["logp_pi", "logp_mu", "ent_pi", "ent_mu", "lse_pi", "lse_mu", "z_pi", "z_mu"]
    out = {k: np.zeros(n_rows, np.float64) for k in names}
    _check(lib().acrl_ref_score(n_rows, d, V, _p(h), _p(w), _p(hq), _p(hs), _p(wq), _p(ws),
                                scaling, _p(ids), _p(m), inv_temperature,
                                *[_p(out[k]) for k in names]), "score")
    return out


def token_divergence(z_pi, z_mu):
    """(KL(pi||mu), KL(mu||pi), Euclidean distance) of softmax(z_pi), softmax(z_mu)."""
    zp = _c(z_pi, np.float64)
    zm = _c(z_mu, np.float64)
    out = np.zeros(3, np.float64)
    lib().acrl_ref_token_divergence(_p(zp), _p(zm), zp.size, _p(out[0:1]), _p(out[1:2]), _p(out[2:3]))
    return float(out[0]), float(out[1]), float(out[2])


def divergence(h, w, hq, hq_scales, wq, wq_scales, scaling: int, mask=None,
               inv_temperature: float = 1.0) -> dict:
    """Full-vocabulary KL(pi||mu), KL(mu||pi) and Euclidean distance of every row."""
    h, w = _c(h, np.uint16), _c(w, np.uint16)
    hq, wq = _c(hq, np.uint8), _c(wq, np.uint8)
    n_rows, d = h.shape
    V = w.shape[0]
    sdt = np.uint8 if scaling == MX32 else np.float32
    hs, ws = _c(hq_scales, sdt), _c(wq_scales, sdt)
    m = None if mask is None else _c(mask, np.uint8)
    out = {k: np.zeros(n_rows, np.float64) for k in ("kl_pi_mu", "kl_mu_pi", "l2")}
    _check(lib().acrl_ref_divergence(n_rows, d, V, _p(h), _p(w), _p(hq), _p(hs), _p(wq), _p(ws), scaling,
                                     _p(m), inv_temperature, _p(out["kl_pi_mu"]), _p(out["kl_mu_pi"]),
                                     _p(out["l2"])), "divergence")
    return out


# ---------------------------------------------------------------- a6/a7
def discrepancy_reduce(B: int, L: int, logp_pi, logp_mu, mask, group_of_seq, n_groups: int,
                       ent_pi=None, ent_mu=None) -> dict:
    lp_p, lp_m = _c(logp_pi, np.float64).reshape(-1), _c(logp_mu, np.float64).reshape(-1)
    ep = None if ent_pi is None else _c(ent_pi, np.float64).reshape(-1)
    em = None if ent_mu is None else _c(ent_mu, np.float64).reshape(-1)
    m = _c(mask, np.uint8).reshape(-1)
    g = _c(group_of_seq, np.int32)
    out = dict(d_tok=np.zeros(B * L), seq_len=np.zeros(B, np.int32), seq_sum_d=np.zeros(B),
               seq_sum_logratio=np.zeros(B), seq_mean_d=np.zeros(B),
               group_y=np.zeros(max(n_groups, 0)), group_nseq=np.zeros(max(n_groups, 0), np.int32),
               stats=np.zeros(N_STATS))
    keys = ["d_tok", "seq_len", "seq_sum_d", "seq_sum_logratio", "seq_mean_d", "group_y",
            "group_nseq", "stats"]
    _check(lib().acrl_ref_discrepancy_reduce(B, L, _p(lp_p), _p(lp_m), _p(ep), _p(em), _p(m),
                                             _p(g), n_groups, *[_p(out[k]) for k in keys]),
           "discrepancy_reduce")
    return out


# ---------------------------------------------------------------- a8
def controller_step(B: int, L: int, mask, group_of_seq, logp_pi, logp_mu, adv,
                    adv_per_token: bool, y_level: int, seq_mean_d, group_y, stats,
                    X: float, gamma: float, C: float, mode: int = 0, k: float = 1.0,
                    n_groups: Optional[int] = None):
    m = _c(mask, np.uint8).reshape(-1)
    g = _c(group_of_seq, np.int32)
    lp_p, lp_m = _c(logp_pi, np.float64).reshape(-1), _c(logp_mu, np.float64).reshape(-1)
    a = _c(adv, np.float64).reshape(-1)
    smd = None if seq_mean_d is None else _c(seq_mean_d, np.float64)
    gy = None if group_y is None else _c(group_y, np.float64)
    st = None if stats is None else _c(stats, np.float64)
    alpha = np.zeros(B * L)
    weight = np.zeros(B * L)
    ng = len(group_y) if (n_groups is None and group_y is not None) else (n_groups or 0)
    _check(lib().acrl_ref_controller_step(B, L, _p(m), _p(g), int(ng), _p(lp_p), _p(lp_m), _p(a),
                                          int(bool(adv_per_token)), y_level, _p(smd), _p(gy),
                                          _p(st), X, gamma, C, int(mode), float(k), _p(alpha),
                                          _p(weight)),
           "controller_step")
    return alpha, weight


def reference_x(group_y, group_nseq) -> float:
    gy = _c(group_y, np.float64)
    gn = _c(group_nseq, np.int32)
    X = np.zeros(1)
    _check(lib().acrl_ref_reference_x(_p(gy), _p(gn), gy.size, _p(X)), "reference_x")
    return float(X[0])


def sample_inverse_cdf(z: np.ndarray, u: np.ndarray) -> np.ndarray:
    z = _c(z, np.float64)
    n_rows, V = z.shape
    u = _c(u, np.float64)
    ids = np.empty(n_rows, np.int32)
    _check(lib().acrl_ref_sample_inverse_cdf(_p(z), n_rows, V, _p(u), _p(ids)), "sample")
    return ids


def philox4x32_10(ctr, key) -> np.ndarray:
    c = np.ascontiguousarray(ctr, np.uint32)
    k = np.ascontiguousarray(key, np.uint32)
    out = np.zeros(4, np.uint32)
    lib().acrl_ref_philox4x32_10(_p(c), _p(k), _p(out))
    return out


def sample_uniform(seed: int, t: int, v: int) -> float:
    return float(lib().acrl_ref_sample_uniform(seed, t, v))


def gumbel_sample(z: np.ndarray, seed: int, row_offset: int = 0):
    """Gumbel-max draw from softmax(z) per row; returns (ids, winning keys)."""
    z = _c(z, np.float64)
    n_rows, V = z.shape
    ids = np.empty(n_rows, np.int32)
    keys = np.empty(n_rows)
    _check(lib().acrl_ref_gumbel_sample(_p(z), n_rows, V, seed, row_offset, _p(ids), _p(keys)),
           "gumbel_sample")
    return ids, keys


def block_gumbel_sample(z: np.ndarray, seed: int, row_offset: int = 0):
    """Blockwise Gumbel-max draw from softmax(z) per row (two uniforms per
    16-row block); returns (ids, winning keys, winning blocks)."""
    z = _c(z, np.float64)
    n_rows, V = z.shape
    ids = np.empty(n_rows, np.int32)
    keys = np.empty(n_rows)
    blocks = np.empty(n_rows, np.int64)
    _check(lib().acrl_ref_block_gumbel_sample(_p(z), n_rows, V, seed, row_offset, _p(ids), _p(keys), _p(blocks)),
           "block_gumbel_sample")
    return ids, keys, blocks


def block_gumbel_keys(z_row: np.ndarray, seed: int, t: int) -> np.ndarray:
    """Every block's key lse_k - ln(-ln u_k) of one token's logits."""
    z = _c(z_row, np.float64)
    keys = np.empty(2 * ((z.size + 31) // 32))
    _check(lib().acrl_ref_block_gumbel_keys(_p(z), z.size, seed, t, _p(keys)), "block_gumbel_keys")
    return keys


def block_pick(z_row: np.ndarray, seed: int, t: int, k: int):
    """(row, cumulative probabilities of the block's 16 slots, u'_k)."""
    z = _c(z_row, np.float64)
    cum = np.empty(16)
    u = np.empty(1)
    row = lib().acrl_ref_block_pick(_p(z), z.size, seed, t, int(k), _p(cum), _p(u))
    return int(row), cum, float(u[0])


def block_slot_rows(k: int, V: int) -> np.ndarray:
    """Rows of block k's 16 slots (-1 past V), in slot order."""
    q = np.arange(16)
    v = 32 * (k // 2) + 8 * (q // 4) + 4 * (k % 2) + q % 4
    return np.where(v < V, v, -1)


def block_of_row(v):
    """Block of vocabulary row v in the blockwise sampler."""
    v = np.asarray(v, np.int64)
    return 2 * (v // 32) + (v // 4) % 2


# ------------------------------------------------- surrogate and backward
def surrogate(B: int, L: int, mask, group_of_seq, n_groups: int, logp_new, logp_old, adv,
              adv_per_token: bool = False, weight=None, eps_low: float = 0.2,
              eps_high: float = 0.2):
    """(coef [B*L], loss): d loss/d logp_new and loss = -J of Eq. ACRL."""
    m = _c(mask, np.uint8).ravel()
    g = _c(group_of_seq, np.int32)
    ln = _c(logp_new, np.float64).ravel()
    lo = _c(logp_old, np.float64).ravel()
    a = _c(adv, np.float64).ravel()
    wt = None if weight is None else _c(weight, np.float64).ravel()
    coef = np.empty(B * L, np.float64)
    loss = np.empty(1, np.float64)
    _check(lib().acrl_ref_surrogate(B, L, _p(m), _p(g), n_groups, _p(ln), _p(lo), _p(a),
                                    int(adv_per_token), _p(wt), eps_low, eps_high, _p(coef),
                                    _p(loss)), "surrogate")
    return coef, float(loss[0])


def lm_head_backward(h, w, ids, coef, inv_temperature: float = 1.0, hrows=None, wrows=None,
                     want_abs: bool = False):
    """Rows of dH = dZ W and dW = dZ^T H (float64), dZ = coef (onehot - p) / tau.

    h: bf16 bits [n, d]; w: bf16 bits [V, d]; hrows / wrows: the rows wanted
    (None = all).  Returns (dh, dw) or, with want_abs, (dh, dw, dh_abs, dw_abs).
    """
    h = _c(h, np.uint16)
    w = _c(w, np.uint16)
    n, d = h.shape
    V = w.shape[0]
    ids = _c(ids, np.int32)
    cf = _c(coef, np.float64)
    hr = np.arange(n, dtype=np.int64) if hrows is None else _c(hrows, np.int64)
    wr = np.arange(V, dtype=np.int64) if wrows is None else _c(wrows, np.int64)
    dh = np.empty((hr.size, d), np.float64)
    dw = np.empty((wr.size, d), np.float64)
    dha = np.empty((hr.size, d), np.float64) if want_abs else None
    dwa = np.empty((wr.size, d), np.float64) if want_abs else None
    _check(lib().acrl_ref_lm_head_backward(n, d, V, _p(h), _p(w), _p(ids), _p(cf), inv_temperature,
                                           hr.size, _p(hr), _p(dh), _p(dha), wr.size, _p(wr), _p(dw),
                                           _p(dwa)), "lm_head_backward")
    return (dh, dw, dha, dwa) if want_abs else (dh, dw)

