"""The C-ABI library loads, exports every symbol include/acrl.h declares, and
rejects out-of-contract arguments on the host (no GPU needed: argument
validation happens before any HIP call)."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "acrl.h")


def _acrl():
    from paper_2607_24062_amd import acrl
    try:
        acrl.lib()
    except (RuntimeError, OSError) as e:  # library not built in this checkout
        pytest.skip("libacrl.so not available: %s" % e)
    return acrl


def _declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(acrl_[a-z0-9_]+)\s*\(", src)))


def test_header_declares_the_four_entry_points():
    names = _declared_functions()
    for n in ("acrl_quantize_fp8", "acrl_score_pi_mu", "acrl_discrepancy_reduce",
              "acrl_controller_step"):
        assert n in names


def test_every_declared_symbol_is_exported():
    acrl = _acrl()
    L = acrl.lib()
    for n in _declared_functions():
        assert hasattr(L, n), n
    assert sorted(acrl.EXPORTED) == _declared_functions()


def test_exported_dynamic_symbols_match_header():
    acrl = _acrl()
    out = subprocess.run(["nm", "-D", "--defined-only", acrl.LIB_PATH], capture_output=True, text=True)
    if out.returncode != 0:
        pytest.skip("nm unavailable")
    syms = sorted(set(re.findall(r"\sT\s(acrl_[a-z0-9_]+)$", out.stdout, flags=re.M)))
    assert syms == _declared_functions()


def test_descriptor_layout_matches_binding():
    acrl = _acrl()
    sizes = [ctypes.c_size_t() for _ in range(6)]
    acrl.lib().acrl_abi_struct_sizes(*[ctypes.byref(s) for s in sizes])
    assert [s.value for s in sizes] == [ctypes.sizeof(acrl.ScoreDesc), ctypes.sizeof(acrl.ReduceDesc),
                                        ctypes.sizeof(acrl.ControllerDesc), ctypes.sizeof(acrl.SampleDesc),
                                        ctypes.sizeof(acrl.SurrogateDesc), ctypes.sizeof(acrl.BackwardDesc)]
    assert acrl.lib().acrl_abi_version() == 6


def test_status_strings():
    acrl = _acrl()
    L = acrl.lib()
    assert L.acrl_status_string(0) == b"ok"
    assert L.acrl_status_string(1) == b"invalid argument"
    assert L.acrl_status_string(99) == b"unknown status"


def _fake(n=16):
    # host buffers standing in for device pointers: never dereferenced,
    # because validation fails before any kernel launch
    return (ctypes.c_uint8 * n)()


def test_quantize_rejects_bad_shapes():
    acrl = _acrl()
    L = acrl.lib()
    buf = _fake(4096)
    p = ctypes.cast(buf, ctypes.c_void_p)
    assert L.acrl_quantize_fp8(p, 4, 33, 33, 1, 0, p, p, None, 0, None) == acrl.ACRL_ERR_INVALID_ARG
    assert b"multiple of 32" in L.acrl_last_error()
    assert L.acrl_quantize_fp8(p, -1, 64, 64, 1, 0, p, p, None, 0, None) == acrl.ACRL_ERR_INVALID_ARG
    assert L.acrl_quantize_fp8(p, 4, 64, 60, 1, 0, p, p, None, 0, None) == acrl.ACRL_ERR_INVALID_ARG
    assert L.acrl_quantize_fp8(p, 4, 64, 64, 7, 0, p, p, None, 0, None) == acrl.ACRL_ERR_INVALID_ARG
    assert L.acrl_quantize_fp8(p, 4, 64, 64, 1, 5, p, p, None, 0, None) == acrl.ACRL_ERR_INVALID_ARG
    # per-tensor needs a workspace
    assert L.acrl_quantize_fp8(p, 4, 64, 64, 0, 0, p, p, None, 0, None) == acrl.ACRL_ERR_WORKSPACE
    nb = ctypes.c_size_t()
    assert L.acrl_quantize_workspace_size(4, 64, 0, ctypes.byref(nb)) == 0 and nb.value > 0
    assert L.acrl_quantize_workspace_size(4, 64, 1, ctypes.byref(nb)) == 0 and nb.value == 0


def test_score_rejects_bad_arguments():
    acrl = _acrl()
    L = acrl.lib()
    buf = _fake(64)
    p = ctypes.c_void_p(ctypes.addressof(buf) + (-ctypes.addressof(buf)) % 16)
    base = dict(n_rows=4, d=256, V=1000, h=p, w=p, hq=p, hq_scales=p, wq=p, wq_scales=p,
                mu_scaling=1, inv_temperature=1.0, token_ids=p, logp_pi=p, logp_mu=p,
                workspace=p, workspace_bytes=1 << 40)
    for bad in (dict(d=100), dict(d=0), dict(V=0), dict(n_rows=-1), dict(mu_scaling=3),
                dict(inv_temperature=0.0), dict(inv_temperature=-1.0), dict(w=None),
                dict(token_ids=None)):
        desc = acrl.ScoreDesc(**{**base, **bad})
        assert L.acrl_score_pi_mu(ctypes.byref(desc), None) == acrl.ACRL_ERR_INVALID_ARG, bad
    desc = acrl.ScoreDesc(**{**base, "workspace_bytes": 16})
    assert L.acrl_score_pi_mu(ctypes.byref(desc), None) == acrl.ACRL_ERR_WORKSPACE
    assert L.acrl_score_pi_mu(None, None) == acrl.ACRL_ERR_INVALID_ARG
    nb = ctypes.c_size_t()
    assert L.acrl_score_workspace_size(300, 256, 1000, 1, ctypes.byref(nb)) == 0
    assert nb.value >= 2 * 3 * 4 * 300


def test_measures_passes_share_the_rows_evenly():
    # 66 token tiles in passes of at most 64 tiles: two passes of 33, so the
    # workspace holds mu's logits of 33 tiles, as for passes of at most 33 or
    # 34 tiles; one pass of all 66 needs more
    L = _acrl().lib()
    rows, tile = 66 * 256, 256

    def ws(chunk):
        nb = ctypes.c_size_t()
        assert L.acrl_score_div_workspace_size(rows, 256, 1000, 1, chunk, ctypes.byref(nb)) == 0
        return nb.value

    assert ws(64 * tile) == ws(33 * tile) == ws(34 * tile) == ws(64 * tile - 5)
    # per pass row: V padded to 1024 logits, mu's lse, five sums per 128 vocabulary rows (4 B each)
    assert ws(66 * tile) - ws(33 * tile) == 33 * tile * (1024 + 1 + 5 * 2 * 4) * 4
    assert ws(0) == ws(16384)


def test_reduce_and_controller_reject_bad_arguments():
    acrl = _acrl()
    L = acrl.lib()
    buf = _fake(64)
    p = ctypes.cast(buf, ctypes.c_void_p)
    desc = acrl.ReduceDesc(B=-1, L=4, n_groups=1, stats=p)
    assert L.acrl_discrepancy_reduce(ctypes.byref(desc), None) == acrl.ACRL_ERR_INVALID_ARG
    desc = acrl.ReduceDesc(B=2, L=4, n_groups=0, logp_pi=p, logp_mu=p, mask=p, group_of_seq=p,
                           seq_mean_d=p, stats=p)
    assert L.acrl_discrepancy_reduce(ctypes.byref(desc), None) == acrl.ACRL_ERR_INVALID_ARG
    desc = acrl.ReduceDesc(B=2, L=4, n_groups=1, logp_pi=p, logp_mu=p, mask=p, group_of_seq=p,
                           seq_mean_d=p, group_y=p, stats=p, workspace=p, workspace_bytes=1)
    assert L.acrl_discrepancy_reduce(ctypes.byref(desc), None) == acrl.ACRL_ERR_WORKSPACE
    ok = dict(B=2, L=4, n_groups=1, mask=p, group_of_seq=p, logp_pi=p, logp_mu=p, adv=p,
              y_level=0, group_y=p, X=0.01, gamma=0.5, C=3.0, weight=p)
    # Sec. 4.1 requires gamma > 0 and C > 1; X > 0 for Y/X to exist
    for bad in (dict(X=0.0), dict(gamma=0.0), dict(C=1.0), dict(C=0.5), dict(X=-1.0),
                dict(y_level=9), dict(group_y=None)):
        d = acrl.ControllerDesc(**{**ok, **bad})
        assert L.acrl_controller_step(ctypes.byref(d), None) == acrl.ACRL_ERR_INVALID_ARG, bad


def test_reference_from_groups_host_helper():
    acrl = _acrl()
    assert abs(acrl.acrl_reference_from_groups([0.01, 0.5, 0.03], [8, 0, 8]) - 0.02) < 1e-8
    with pytest.raises(acrl.AcrlError):
        acrl.acrl_reference_from_groups([0.01], [0])


def test_surrogate_rejects_bad_arguments():
    acrl = _acrl()
    L = acrl.lib()
    buf = _fake(64)
    p = ctypes.cast(buf, ctypes.c_void_p)
    ok = dict(B=2, L=4, n_groups=1, mask=p, group_of_seq=p, logp_new=p, logp_old=p, adv=p,
              eps_low=0.2, eps_high=0.2, coef=p, loss=p, workspace=p, workspace_bytes=1 << 30)
    for bad in (dict(B=-1), dict(n_groups=0), dict(eps_low=1.0), dict(eps_low=-0.1), dict(eps_high=-0.1),
                dict(loss=None), dict(coef=None), dict(logp_old=None)):
        d = acrl.SurrogateDesc(**{**ok, **bad})
        assert L.acrl_surrogate(ctypes.byref(d), None) == acrl.ACRL_ERR_INVALID_ARG, bad
    d = acrl.SurrogateDesc(**{**ok, "workspace_bytes": 1})
    assert L.acrl_surrogate(ctypes.byref(d), None) == acrl.ACRL_ERR_WORKSPACE
    nb = ctypes.c_size_t()
    assert L.acrl_surrogate_workspace_size(64, 8, ctypes.byref(nb)) == 0 and nb.value >= 64 * 16


def test_backward_rejects_bad_arguments():
    acrl = _acrl()
    L = acrl.lib()
    buf = _fake(64)
    p = ctypes.c_void_p(ctypes.addressof(buf) + (-ctypes.addressof(buf)) % 16)
    ok = dict(n_rows=4, d=256, V=1000, h=p, w=p, token_ids=p, coef=p, lse=p, inv_temperature=1.0,
              dh=p, dw=p, workspace=p, workspace_bytes=1 << 40)
    for bad in (dict(d=100), dict(V=0), dict(V=1 << 23), dict(n_rows=-1), dict(inv_temperature=0.0),
                dict(dh=None, dw=None), dict(lse=None), dict(coef=None), dict(token_chunk=-5)):
        d = acrl.BackwardDesc(**{**ok, **bad})
        assert L.acrl_lm_head_backward(ctypes.byref(d), None) == acrl.ACRL_ERR_INVALID_ARG, bad
    d = acrl.BackwardDesc(**{**ok, "workspace_bytes": 16})
    assert L.acrl_lm_head_backward(ctypes.byref(d), None) == acrl.ACRL_ERR_WORKSPACE
    nb = ctypes.c_size_t()
    assert L.acrl_backward_workspace_size(300, 256, 1000, 0, ctypes.byref(nb)) == 0
    # W, W^T, H, H^T and the two dZ images of one 512-row chunk
    assert nb.value >= 2 * (1024 * 256 * 2) + 2 * (512 * 256 * 2) + 2 * (512 * 1024 * 2)
