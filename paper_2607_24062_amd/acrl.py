"""Thin Python binding of libacrl (ctypes).

Every entry point of include/acrl.h is exposed under the same name; the
wrappers only marshal arguments (torch tensors supply device memory, the
current torch stream supplies the HIP stream).  All computation runs in the
library's HIP kernels.  If libacrl.so is missing or cannot be loaded, every
call raises: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libacrl.so")

ACRL_OK, ACRL_ERR_INVALID_ARG, ACRL_ERR_UNSUPPORTED, ACRL_ERR_WORKSPACE, ACRL_ERR_HIP = range(5)
SCALE_PER_TENSOR, SCALE_PER_ROW, SCALE_MX32 = 0, 1, 2
ROUND_NEAREST_EVEN, ROUND_TOWARD_ZERO = 0, 1
Y_GROUP, Y_SEQUENCE, Y_BATCH = 0, 1, 2
CTRL_ACRL, CTRL_TIS, CTRL_MIS, CTRL_CONTINUOUS, CTRL_FALLBACK = 0, 1, 2, 3, 4
POLICY_BOTH, POLICY_PI, POLICY_MU = 0, 1, 2
N_STATS = 10
STAT_NAMES = ["y_batch", "tok_mean_d", "tok_max_d", "tok_std_d", "mean_h_pi", "mean_h_mu",
              "n_tokens", "n_groups", "tok_mean_logratio", "n_seqs"]

EXPORTED = [
    "acrl_status_string", "acrl_last_error", "acrl_abi_version", "acrl_abi_struct_sizes",
    "acrl_quantize_workspace_size", "acrl_quantize_fp8", "acrl_fp8_encode",
    "acrl_score_workspace_size", "acrl_score_div_workspace_size", "acrl_score_workspace_query", "acrl_score_pi_mu",
    "acrl_packed_weights_size", "acrl_pack_weights",
    "acrl_reduce_workspace_size", "acrl_discrepancy_reduce", "acrl_discrepancy_reduce_noalloc",
    "acrl_controller_step", "acrl_reference_from_groups", "acrl_sample_mu",
    "acrl_surrogate_workspace_size", "acrl_surrogate",
    "acrl_backward_workspace_size", "acrl_lm_head_backward",
]

_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_I32 = ctypes.c_int32
_F32 = ctypes.c_float
_SZ = ctypes.c_size_t


class ScoreDesc(ctypes.Structure):
    _fields_ = [("n_rows", _I64), ("d", _I64), ("V", _I64),
                ("h", _P), ("w", _P), ("hq", _P), ("hq_scales", _P), ("wq", _P), ("wq_scales", _P),
                ("mu_scaling", _I32), ("inv_temperature", _F32),
                ("token_ids", _P), ("mask", _P), ("out_slot", _P),
                ("logp_pi", _P), ("logp_mu", _P), ("entropy_pi", _P), ("entropy_mu", _P),
                ("lse_pi", _P), ("lse_mu", _P), ("logit_pi", _P), ("logit_mu", _P),
                ("error_flag", _P), ("workspace", _P), ("workspace_bytes", _SZ),
                ("kl_pi_mu", _P), ("kl_mu_pi", _P), ("l2", _P), ("div_chunk", _I64),
                ("policies", _I32), ("packed_weights", _P), ("packed_weights_bytes", _SZ)]


class ReduceDesc(ctypes.Structure):
    _fields_ = [("B", _I64), ("L", _I64), ("n_groups", _I64),
                ("logp_pi", _P), ("logp_mu", _P), ("entropy_pi", _P), ("entropy_mu", _P),
                ("mask", _P), ("group_of_seq", _P),
                ("d_tok", _P), ("seq_len", _P), ("seq_sum_d", _P), ("seq_sum_logratio", _P),
                ("seq_mean_d", _P), ("group_y", _P), ("group_nseq", _P), ("stats", _P),
                ("workspace", _P), ("workspace_bytes", _SZ)]


class ControllerDesc(ctypes.Structure):
    _fields_ = [("B", _I64), ("L", _I64), ("n_groups", _I64),
                ("mask", _P), ("group_of_seq", _P), ("logp_pi", _P), ("logp_mu", _P),
                ("adv", _P), ("adv_per_token", _I32), ("y_level", _I32),
                ("seq_mean_d", _P), ("group_y", _P), ("stats", _P),
                ("X", _F32), ("gamma", _F32), ("C", _F32),
                ("alpha", _P), ("weight", _P), ("mode", _I32), ("k", _F32),
                ("seq_sum_logratio", _P)]


class SurrogateDesc(ctypes.Structure):
    _fields_ = [("B", _I64), ("L", _I64), ("n_groups", _I64),
                ("mask", _P), ("group_of_seq", _P), ("logp_new", _P), ("logp_old", _P),
                ("adv", _P), ("adv_per_token", _I32), ("eps_low", _F32), ("eps_high", _F32),
                ("weight", _P), ("coef", _P), ("loss", _P), ("workspace", _P), ("workspace_bytes", _SZ)]


class BackwardDesc(ctypes.Structure):
    _fields_ = [("n_rows", _I64), ("d", _I64), ("V", _I64), ("h", _P), ("w", _P),
                ("token_ids", _P), ("row_slot", _P), ("coef", _P), ("lse", _P),
                ("inv_temperature", _F32), ("dh", _P), ("dw", _P), ("accumulate_dw", _I32),
                ("token_chunk", _I64), ("workspace", _P), ("workspace_bytes", _SZ)]


class SampleDesc(ctypes.Structure):
    _fields_ = [("n_rows", _I64), ("d", _I64), ("V", _I64),
                ("hq", _P), ("hq_scales", _P), ("wq", _P), ("wq_scales", _P),
                ("mu_scaling", _I32), ("inv_temperature", _F32),
                ("seed", ctypes.c_uint64), ("row_offset", _I64),
                ("ids", _P), ("logp_mu", _P), ("workspace", _P), ("workspace_bytes", _SZ),
                ("packed_weights", _P), ("packed_weights_bytes", _SZ)]


class AcrlError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__("%s failed: %s (%s)" % (where, _status_names.get(status, status), detail))
        self.status = status


_status_names = {0: "ok", 1: "invalid argument", 2: "unsupported", 3: "workspace too small",
                 4: "HIP runtime error"}

_lib: Optional[ctypes.CDLL] = None


def lib() -> ctypes.CDLL:
    """Load libacrl.so (built in-tree by paper_2607_24062_amd.build)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libacrl.so is not built (%s); run python -m paper_2607_24062_amd.build"
                               % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        L.acrl_status_string.restype = ctypes.c_char_p
        L.acrl_status_string.argtypes = [_I32]
        L.acrl_last_error.restype = ctypes.c_char_p
        L.acrl_last_error.argtypes = []
        L.acrl_abi_version.restype = _I32
        L.acrl_abi_struct_sizes.restype = None
        L.acrl_abi_struct_sizes.argtypes = [ctypes.POINTER(_SZ)] * 6
        L.acrl_quantize_workspace_size.restype = _I32
        L.acrl_quantize_workspace_size.argtypes = [_I64, _I64, _I32, ctypes.POINTER(_SZ)]
        L.acrl_quantize_fp8.restype = _I32
        L.acrl_quantize_fp8.argtypes = [_P, _I64, _I64, _I64, _I32, _I32, _P, _P, _P, _SZ, _P]
        L.acrl_fp8_encode.restype = _I32
        L.acrl_fp8_encode.argtypes = [_P, _I64, _I32, _P, _P]
        L.acrl_score_workspace_size.restype = _I32
        L.acrl_score_workspace_size.argtypes = [_I64, _I64, _I64, _I32, ctypes.POINTER(_SZ)]
        L.acrl_score_div_workspace_size.restype = _I32
        L.acrl_score_div_workspace_size.argtypes = [_I64, _I64, _I64, _I32, _I64, ctypes.POINTER(_SZ)]
        L.acrl_score_pi_mu.restype = _I32
        L.acrl_score_pi_mu.argtypes = [ctypes.POINTER(ScoreDesc), _P]
        L.acrl_score_workspace_query.restype = _I32
        L.acrl_score_workspace_query.argtypes = [ctypes.POINTER(ScoreDesc), ctypes.POINTER(_SZ)]
        L.acrl_packed_weights_size.restype = _I32
        L.acrl_packed_weights_size.argtypes = [_I64, _I64, _I32, ctypes.POINTER(_SZ)]
        L.acrl_pack_weights.restype = _I32
        L.acrl_pack_weights.argtypes = [_P, _P, _P, _I64, _I64, _I32, _P, _SZ, _P]
        L.acrl_reduce_workspace_size.restype = _I32
        L.acrl_reduce_workspace_size.argtypes = [_I64, _I64, _I64, ctypes.POINTER(_SZ)]
        L.acrl_discrepancy_reduce.restype = _I32
        L.acrl_discrepancy_reduce.argtypes = [ctypes.POINTER(ReduceDesc), _P]
        L.acrl_discrepancy_reduce_noalloc.restype = _I32
        L.acrl_discrepancy_reduce_noalloc.argtypes = [ctypes.POINTER(ReduceDesc), _P]
        L.acrl_controller_step.restype = _I32
        L.acrl_controller_step.argtypes = [ctypes.POINTER(ControllerDesc), _P]
        L.acrl_reference_from_groups.restype = _I32
        L.acrl_reference_from_groups.argtypes = [_P, _P, _I64, ctypes.POINTER(_F32)]
        L.acrl_sample_mu.restype = _I32
        L.acrl_sample_mu.argtypes = [ctypes.POINTER(SampleDesc), _P]
        L.acrl_surrogate_workspace_size.restype = _I32
        L.acrl_surrogate_workspace_size.argtypes = [_I64, _I64, ctypes.POINTER(_SZ)]
        L.acrl_surrogate.restype = _I32
        L.acrl_surrogate.argtypes = [ctypes.POINTER(SurrogateDesc), _P]
        L.acrl_backward_workspace_size.restype = _I32
        L.acrl_backward_workspace_size.argtypes = [_I64, _I64, _I64, _I64, ctypes.POINTER(_SZ)]
        L.acrl_lm_head_backward.restype = _I32
        L.acrl_lm_head_backward.argtypes = [ctypes.POINTER(BackwardDesc), _P]
        sizes = [_SZ() for _ in range(6)]
        L.acrl_abi_struct_sizes(*[ctypes.byref(s) for s in sizes])
        want = [ctypes.sizeof(ScoreDesc), ctypes.sizeof(ReduceDesc), ctypes.sizeof(ControllerDesc),
                ctypes.sizeof(SampleDesc), ctypes.sizeof(SurrogateDesc), ctypes.sizeof(BackwardDesc)]
        got = [s.value for s in sizes]
        if got != want:
            raise RuntimeError("libacrl descriptor layout mismatch: library %s, binding %s" % (got, want))
        _lib = L
    return _lib


def _check(status: int, where: str) -> None:
    if status != ACRL_OK:
        raise AcrlError(status, where, lib().acrl_last_error().decode(errors="replace"))


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _dev(t: torch.Tensor, dtype, name: str):
    if not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if t.dtype != dtype:
        raise ValueError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    return t


_ws_cache: Dict[tuple, torch.Tensor] = {}


def _workspace(nbytes: int, device, stream=None) -> torch.Tensor:
    """A cached device byte buffer of at least nbytes for calls on `stream`
    (the current stream if None), grown on demand.  One buffer per (device,
    stream): calls on one stream run in order, so they may share it, and a
    buffer is allocated on the stream that uses it, so torch's allocator
    recycles a replaced one only after that stream's earlier work."""
    s = stream if stream is not None else torch.cuda.current_stream(device)
    key = (torch.device(device), s.cuda_stream)
    buf = _ws_cache.get(key)
    if buf is None or buf.numel() < nbytes:
        _ws_cache.pop(key, None)
        with torch.cuda.stream(s):
            buf = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
        _ws_cache[key] = buf
    return buf


# ------------------------------------------------------------------ a1/a2
def acrl_quantize_fp8(x: torch.Tensor, scaling: int, rounding: int = ROUND_NEAREST_EVEN,
                      q: Optional[torch.Tensor] = None, scales: Optional[torch.Tensor] = None,
                      stream=None):
    """x: bf16 [rows, cols] -> (q uint8 [rows, cols], scales).  x may be a
    column slice of a wider matrix (unit column stride, row stride = ld)."""
    if x.dim() != 2:
        raise ValueError("x must be 2-D")
    rows, cols = x.shape
    if x.is_contiguous():
        _dev(x, torch.bfloat16, "x")
        ld = cols
    else:
        if not x.is_cuda or x.dtype != torch.bfloat16 or x.stride(1) != 1 or x.stride(0) < cols:
            raise ValueError("x must be a bf16 device matrix with unit column stride")
        ld = x.stride(0)
    if q is None:
        q = torch.empty((rows, cols), dtype=torch.uint8, device=x.device)
    if scales is None:
        if scaling == SCALE_PER_TENSOR:
            scales = torch.empty(1, dtype=torch.float32, device=x.device)
        elif scaling == SCALE_PER_ROW:
            scales = torch.empty(rows, dtype=torch.float32, device=x.device)
        else:
            scales = torch.empty((rows, cols // 32), dtype=torch.uint8, device=x.device)
    nb = _SZ()
    _check(lib().acrl_quantize_workspace_size(rows, cols, scaling, ctypes.byref(nb)),
           "acrl_quantize_workspace_size")
    ws = _workspace(nb.value, x.device, stream) if nb.value else None
    _check(lib().acrl_quantize_fp8(_ptr(x), rows, cols, ld, scaling, rounding, _ptr(q), _ptr(scales),
                                   _ptr(ws), nb.value, _stream(stream)), "acrl_quantize_fp8")
    return q, scales


def acrl_fp8_encode(x: torch.Tensor, rounding: int = ROUND_NEAREST_EVEN, q=None, stream=None):
    _dev(x, torch.float32, "x")
    if q is None:
        q = torch.empty(x.shape, dtype=torch.uint8, device=x.device)
    _check(lib().acrl_fp8_encode(_ptr(x), x.numel(), rounding, _ptr(q), _stream(stream)),
           "acrl_fp8_encode")
    return q


# ------------------------------------------------------------------ a3..a5
def acrl_pack_weights(w, wq, wq_scales, mu_scaling: int, packed=None, stream=None):
    """The tiled copy of W and Wq (and Wq's MX scales) the scorers stream
    from, once per weight version; returns the uint8 device buffer to pass
    as packed_weights."""
    _dev(w, torch.bfloat16, "w")
    _dev(wq, torch.uint8, "wq")
    V, d = w.shape
    nb = _SZ()
    _check(lib().acrl_packed_weights_size(V, d, mu_scaling, ctypes.byref(nb)), "acrl_packed_weights_size")
    if packed is None:
        packed = torch.empty(nb.value, dtype=torch.uint8, device=w.device)
    _check(lib().acrl_pack_weights(_ptr(w), _ptr(wq), _ptr(wq_scales), V, d, mu_scaling, _ptr(packed),
                                   packed.numel(), _stream(stream)), "acrl_pack_weights")
    return packed


def acrl_score_pi_mu(h, w, hq, hq_scales, wq, wq_scales, mu_scaling: int, token_ids,
                     inv_temperature: float = 1.0, mask=None, out_slot=None, n_slots=None,
                     outputs: Optional[dict] = None, want=("entropy", "lse", "logit"),
                     error_flag=None, stream=None, divergence: bool = False, div_chunk: int = 0,
                     policies: int = POLICY_BOTH, packed_weights=None) -> dict:
    """Score every row of h under pi (bf16) and mu (fp8/mxfp8).

    Returns a dict of float32 [n_slots] tensors: logp_pi, logp_mu and, per
    `want`, entropy_pi/mu, lse_pi/mu, logit_pi/mu; with divergence=True also
    the full-vocabulary kl_pi_mu, kl_mu_pi and l2.  Pass `outputs` to reuse
    preallocated tensors.  policies = POLICY_PI / POLICY_MU scores one
    policy only (the other's outputs are left untouched); packed_weights is
    the buffer acrl_pack_weights returned for these w, wq."""
    _dev(h, torch.bfloat16, "h")
    _dev(w, torch.bfloat16, "w")
    _dev(hq, torch.uint8, "hq")
    _dev(wq, torch.uint8, "wq")
    _dev(token_ids, torch.int32, "token_ids")
    n_rows, d = h.shape
    V = w.shape[0]
    if n_slots is None:
        n_slots = n_rows
    dev = h.device
    out = {} if outputs is None else dict(outputs)
    names = ["logp_pi", "logp_mu"]
    for k in want:
        names += [k + "_pi", k + "_mu"]
    if divergence:
        names += ["kl_pi_mu", "kl_mu_pi", "l2"]
    for k in names:
        if k not in out:
            out[k] = torch.zeros(n_slots, dtype=torch.float32, device=dev)
    desc = ScoreDesc(n_rows=n_rows, d=d, V=V, h=_ptr(h), w=_ptr(w), hq=_ptr(hq),
                     hq_scales=_ptr(hq_scales), wq=_ptr(wq), wq_scales=_ptr(wq_scales),
                     mu_scaling=mu_scaling, inv_temperature=float(inv_temperature),
                     token_ids=_ptr(token_ids), mask=_ptr(mask), out_slot=_ptr(out_slot),
                     logp_pi=_ptr(out["logp_pi"]), logp_mu=_ptr(out["logp_mu"]),
                     entropy_pi=_ptr(out.get("entropy_pi")), entropy_mu=_ptr(out.get("entropy_mu")),
                     lse_pi=_ptr(out.get("lse_pi")), lse_mu=_ptr(out.get("lse_mu")),
                     logit_pi=_ptr(out.get("logit_pi")), logit_mu=_ptr(out.get("logit_mu")),
                     error_flag=_ptr(error_flag),
                     kl_pi_mu=_ptr(out.get("kl_pi_mu") if divergence else None),
                     kl_mu_pi=_ptr(out.get("kl_mu_pi") if divergence else None),
                     l2=_ptr(out.get("l2") if divergence else None), div_chunk=int(div_chunk),
                     policies=int(policies), packed_weights=_ptr(packed_weights),
                     packed_weights_bytes=0 if packed_weights is None else packed_weights.numel())
    nb = _SZ()
    _check(lib().acrl_score_workspace_query(ctypes.byref(desc), ctypes.byref(nb)), "acrl_score_workspace_query")
    ws = _workspace(nb.value, dev, stream)
    desc.workspace, desc.workspace_bytes = _ptr(ws), nb.value
    _check(lib().acrl_score_pi_mu(ctypes.byref(desc), _stream(stream)), "acrl_score_pi_mu")
    return out


def acrl_sample_mu(hq, hq_scales, wq, wq_scales, mu_scaling: int, seed: int, row_offset: int = 0,
                   inv_temperature: float = 1.0, ids=None, logp_mu=None, want_logp: bool = True,
                   stream=None, packed_weights=None):
    """Draw one token per row of hq from mu (Gumbel-max in the mu kernel).

    Returns (ids int32 [n_rows], logp_mu float32 [n_rows] or None)."""
    _dev(hq, torch.uint8, "hq")
    _dev(wq, torch.uint8, "wq")
    n_rows, d = hq.shape
    V = wq.shape[0]
    dev = hq.device
    if ids is None:
        ids = torch.empty(n_rows, dtype=torch.int32, device=dev)
    if logp_mu is None and want_logp:
        logp_mu = torch.empty(n_rows, dtype=torch.float32, device=dev)
    nb = _SZ()
    probe = ScoreDesc(n_rows=n_rows, d=d, V=V, mu_scaling=mu_scaling, packed_weights=_ptr(packed_weights))
    _check(lib().acrl_score_workspace_query(ctypes.byref(probe), ctypes.byref(nb)), "acrl_score_workspace_query")
    ws = _workspace(nb.value, dev, stream)
    desc = SampleDesc(n_rows=n_rows, d=d, V=V, hq=_ptr(hq), hq_scales=_ptr(hq_scales), wq=_ptr(wq),
                      wq_scales=_ptr(wq_scales), mu_scaling=mu_scaling,
                      inv_temperature=float(inv_temperature), seed=int(seed) & (2 ** 64 - 1),
                      row_offset=int(row_offset), ids=_ptr(ids), logp_mu=_ptr(logp_mu),
                      workspace=_ptr(ws), workspace_bytes=nb.value, packed_weights=_ptr(packed_weights),
                      packed_weights_bytes=0 if packed_weights is None else packed_weights.numel())
    _check(lib().acrl_sample_mu(ctypes.byref(desc), _stream(stream)), "acrl_sample_mu")
    return ids, logp_mu


# ------------------------------------------------------------------ a6/a7
def _reduce(fn_name: str, B: int, L: int, n_groups: int, logp_pi, logp_mu, mask, group_of_seq,
            entropy_pi, entropy_mu, want_d_tok: bool, stream, use_workspace: bool, out=None) -> dict:
    dev = logp_pi.device
    if out is None:
        out = dict(
            d_tok=torch.empty(B * L, dtype=torch.float32, device=dev) if want_d_tok else None,
            seq_len=torch.empty(B, dtype=torch.int32, device=dev),
            seq_sum_d=torch.empty(B, dtype=torch.float64, device=dev),
            seq_sum_logratio=torch.empty(B, dtype=torch.float64, device=dev),
            seq_mean_d=torch.empty(B, dtype=torch.float32, device=dev),
            group_y=torch.empty(n_groups, dtype=torch.float32, device=dev),
            group_nseq=torch.empty(n_groups, dtype=torch.int32, device=dev),
            stats=torch.empty(N_STATS, dtype=torch.float64, device=dev),
        )
    ws = None
    nbytes = 0
    if use_workspace:
        nb = _SZ()
        _check(lib().acrl_reduce_workspace_size(B, L, n_groups, ctypes.byref(nb)), "acrl_reduce_workspace_size")
        ws = _workspace(nb.value, dev, stream)
        nbytes = nb.value
    desc = ReduceDesc(B=B, L=L, n_groups=n_groups, logp_pi=_ptr(logp_pi), logp_mu=_ptr(logp_mu),
                      entropy_pi=_ptr(entropy_pi), entropy_mu=_ptr(entropy_mu), mask=_ptr(mask),
                      group_of_seq=_ptr(group_of_seq), d_tok=_ptr(out["d_tok"]),
                      seq_len=_ptr(out["seq_len"]), seq_sum_d=_ptr(out["seq_sum_d"]),
                      seq_sum_logratio=_ptr(out["seq_sum_logratio"]), seq_mean_d=_ptr(out["seq_mean_d"]),
                      group_y=_ptr(out["group_y"]), group_nseq=_ptr(out["group_nseq"]),
                      stats=_ptr(out["stats"]), workspace=_ptr(ws), workspace_bytes=nbytes)
    _check(getattr(lib(), fn_name)(ctypes.byref(desc), _stream(stream)), fn_name)
    return out


def acrl_discrepancy_reduce(B: int, L: int, n_groups: int, logp_pi, logp_mu, mask, group_of_seq,
                            entropy_pi=None, entropy_mu=None, want_d_tok: bool = True,
                            stream=None) -> dict:
    """Per-token d, per-response / per-group / batch reductions (a6/a7).
    Returns a dict of device tensors (d_tok, seq_len, seq_sum_d,
    seq_sum_logratio, seq_mean_d, group_y, group_nseq, stats)."""
    return _reduce("acrl_discrepancy_reduce", B, L, n_groups, logp_pi, logp_mu, mask, group_of_seq,
                   entropy_pi, entropy_mu, want_d_tok, stream, True)


def acrl_discrepancy_reduce_noalloc(B: int, L: int, n_groups: int, logp_pi, logp_mu, mask, group_of_seq,
                                    entropy_pi=None, entropy_mu=None, want_d_tok: bool = True,
                                    stream=None, out: Optional[dict] = None) -> dict:
    """The same reduce on the library's fixed per-device scratch (no
    workspace).  With `out` (a dict of preallocated output tensors as
    acrl_discrepancy_reduce returns) nothing is allocated on this path."""
    return _reduce("acrl_discrepancy_reduce_noalloc", B, L, n_groups, logp_pi, logp_mu, mask, group_of_seq,
                   entropy_pi, entropy_mu, want_d_tok, stream, False, out)


# ------------------------------------------------------------------ a8
def acrl_controller_step(B: int, L: int, n_groups: int, mask, group_of_seq, logp_pi, logp_mu, adv,
                         adv_per_token: bool, y_level: int, seq_mean_d, group_y, stats,
                         X: float, gamma: float, C: float, want_alpha: bool = True, stream=None,
                         mode: int = 0, k: float = 1.0, seq_sum_logratio=None):
    dev = logp_pi.device
    alpha = torch.empty(B * L, dtype=torch.float32, device=dev) if want_alpha else None
    weight = torch.empty(B * L, dtype=torch.float32, device=dev)
    desc = ControllerDesc(B=B, L=L, n_groups=n_groups, mask=_ptr(mask), group_of_seq=_ptr(group_of_seq),
                          logp_pi=_ptr(logp_pi), logp_mu=_ptr(logp_mu), adv=_ptr(adv),
                          adv_per_token=int(bool(adv_per_token)), y_level=y_level,
                          seq_mean_d=_ptr(seq_mean_d), group_y=_ptr(group_y), stats=_ptr(stats),
                          X=float(X), gamma=float(gamma), C=float(C), alpha=_ptr(alpha),
                          weight=_ptr(weight), mode=int(mode), k=float(k),
                          seq_sum_logratio=_ptr(seq_sum_logratio))
    _check(lib().acrl_controller_step(ctypes.byref(desc), _stream(stream)), "acrl_controller_step")
    return alpha, weight


def acrl_reference_from_groups(group_y, group_nseq) -> float:
    """Host helper: X = mean of Y_g over non-empty groups (host arrays)."""
    import numpy as np
    gy = np.ascontiguousarray(group_y, np.float32)
    gn = np.ascontiguousarray(group_nseq, np.int32)
    X = _F32()
    _check(lib().acrl_reference_from_groups(gy.ctypes.data_as(_P), gn.ctypes.data_as(_P), gy.size,
                                            ctypes.byref(X)), "acrl_reference_from_groups")
    return float(X.value)


# ------------------------------------------------------------------ surrogate and its backward
def acrl_surrogate(B: int, L: int, n_groups: int, mask, group_of_seq, logp_new, logp_old, adv,
                   adv_per_token: bool, eps_low: float = 0.2, eps_high: float = 0.2, weight=None,
                   coef=None, stream=None):
    """ACRL-weighted clipped surrogate: returns (coef float32 [B*L], loss float64 [1])."""
    dev = logp_new.device
    if coef is None:
        coef = torch.empty(B * L, dtype=torch.float32, device=dev)
    loss = torch.empty(1, dtype=torch.float64, device=dev)
    nb = _SZ()
    _check(lib().acrl_surrogate_workspace_size(B, n_groups, ctypes.byref(nb)), "acrl_surrogate_workspace_size")
    ws = _workspace(nb.value, dev, stream)
    desc = SurrogateDesc(B=B, L=L, n_groups=n_groups, mask=_ptr(mask), group_of_seq=_ptr(group_of_seq),
                         logp_new=_ptr(logp_new), logp_old=_ptr(logp_old), adv=_ptr(adv),
                         adv_per_token=int(bool(adv_per_token)), eps_low=float(eps_low),
                         eps_high=float(eps_high), weight=_ptr(weight), coef=_ptr(coef), loss=_ptr(loss),
                         workspace=_ptr(ws), workspace_bytes=nb.value)
    _check(lib().acrl_surrogate(ctypes.byref(desc), _stream(stream)), "acrl_surrogate")
    return coef, loss


def acrl_lm_head_backward(h, w, token_ids, coef, lse, inv_temperature: float = 1.0, row_slot=None,
                          want_dh: bool = True, want_dw: bool = True, dh=None, dw=None,
                          accumulate_dw: bool = False, token_chunk: int = 0, stream=None):
    """Gradient of the surrogate w.r.t. h [n_rows, d] and w [V, d] (bf16):
    returns (dh float32 [n_rows, d] or None, dw float32 [V, d] or None)."""
    _dev(h, torch.bfloat16, "h")
    _dev(w, torch.bfloat16, "w")
    _dev(token_ids, torch.int32, "token_ids")
    _dev(coef, torch.float32, "coef")
    _dev(lse, torch.float32, "lse")
    n_rows, d = h.shape
    V = w.shape[0]
    dev = h.device
    if want_dh and dh is None:
        dh = torch.empty((n_rows, d), dtype=torch.float32, device=dev)
    if want_dw and dw is None:
        dw = torch.empty((V, d), dtype=torch.float32, device=dev)
    nb = _SZ()
    _check(lib().acrl_backward_workspace_size(n_rows, d, V, int(token_chunk), ctypes.byref(nb)),
           "acrl_backward_workspace_size")
    ws = _workspace(nb.value, dev, stream)
    desc = BackwardDesc(n_rows=n_rows, d=d, V=V, h=_ptr(h), w=_ptr(w), token_ids=_ptr(token_ids),
                        row_slot=_ptr(row_slot), coef=_ptr(coef), lse=_ptr(lse),
                        inv_temperature=float(inv_temperature), dh=_ptr(dh if want_dh else None),
                        dw=_ptr(dw if want_dw else None), accumulate_dw=int(bool(accumulate_dw)),
                        token_chunk=int(token_chunk), workspace=_ptr(ws), workspace_bytes=nb.value)
    _check(lib().acrl_lm_head_backward(ctypes.byref(desc), _stream(stream)), "acrl_lm_head_backward")
    return (dh if want_dh else None), (dw if want_dw else None)
