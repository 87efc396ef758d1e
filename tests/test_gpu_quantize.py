"""GPU parity of acrl_quantize_fp8 / acrl_fp8_encode with the oracle: bit-exact
codes and scales (per-tensor, per-row, MX32; nearest-even and toward-zero)."""
import numpy as np
import pytest

import inputs
import oracle
from cases import random_bf16
from gpu_util import down, torch_dev, up, up_bf16

pytestmark = pytest.mark.gpu

SCHEMES = [(oracle.PER_TENSOR, "tensor"), (oracle.PER_ROW, "row"), (oracle.MX32, "mx")]
ROUNDINGS = [oracle.ROUND_NEAREST_EVEN, oracle.ROUND_TOWARD_ZERO]


def _gpu_quant(x_bits, scaling, rounding):
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    x = up_bf16(torch, dev, x_bits)
    q, s = acrl.acrl_quantize_fp8(x, scaling, rounding)
    torch.cuda.synchronize()
    return down(q), down(s)


def _assert_same(x_bits, scaling, rounding):
    q, s = _gpu_quant(x_bits, scaling, rounding)
    qo, so = oracle.quantize_fp8(x_bits, scaling, rounding)
    assert np.array_equal(s.view(np.uint8), so.view(np.uint8)), "scales differ"
    bad = np.argwhere(q != qo)
    assert bad.size == 0, "codes differ at %s: gpu %s oracle %s" % (
        bad[:5].tolist(), q[tuple(bad[0])] if bad.size else None, qo[tuple(bad[0])] if bad.size else None)


@pytest.mark.parametrize("scaling,tag", SCHEMES)
@pytest.mark.parametrize("rounding", ROUNDINGS)
def test_small_workload_tensors(scaling, tag, rounding):
    w = inputs.WORKLOADS["tiny"]
    _assert_same(inputs.hidden_bf16(w), scaling, rounding)
    _assert_same(inputs.weights_bf16(w), scaling, rounding)


@pytest.mark.parametrize("scaling,tag", SCHEMES)
@pytest.mark.parametrize("shape", [(1, 32), (3, 96), (5, 4096), (7, 8192 + 512), (2, 9000 // 32 * 32)])
def test_shapes_and_register_fallback(scaling, tag, shape):
    # cols > 8192 exercises the per-row kernel's non-register path
    _assert_same(random_bf16(shape, sum(shape), std=2.0), scaling, oracle.ROUND_NEAREST_EVEN)


@pytest.mark.parametrize("scaling,tag", SCHEMES)
def test_edge_values(scaling, tag):
    # every finite bf16 pattern (subnormals, +-0, the largest values), rows of zeros
    b = np.arange(65536, dtype=np.uint32)
    f = (b << 16).view(np.float32)
    bits = b[np.isfinite(f)].astype(np.uint16)
    bits = np.concatenate([bits, np.zeros(64 * 32 - bits.size % (64 * 32), np.uint16)])
    x = bits.reshape(-1, 64 * 32)
    x[3] = 0          # an all-zero row (scale 1 / E8M0 code 0)
    x[4, :] = 0x8000  # negative zeros
    for rounding in ROUNDINGS:
        _assert_same(x, scaling, rounding)


def _all_magnitudes_up_to(amax_bits):
    """Every bf16 x with |x| <= amax, both signs (amax itself included)."""
    b = np.arange(0x7F80, dtype=np.uint16)
    b = b[b <= amax_bits]
    return np.concatenate([b, b | 0x8000]).astype(np.uint16)


# bf16 amax patterns: subnormal, far below / just below / at / just above
# 2^-64 (where the row kernel switches from the divide to the reciprocal
# path), 1, 448, the largest finite value
AMAX_BITS = [0x0001, 0x0C5A, 0x1F7F, 0x1F80, 0x1F81, 0x2A3B, 0x3F80, 0x43E0, 0x5555, 0x7F7F]


@pytest.mark.parametrize("rounding", ROUNDINGS)
def test_division_paths_every_magnitude(rounding):
    # per-row: each row holds every magnitude up to its amax, so both division
    # paths see every input they can get
    rows = [_all_magnitudes_up_to(a) for a in AMAX_BITS]
    cols = (max(r.size for r in rows) + 31) // 32 * 32
    x = np.zeros((len(rows), cols), np.uint16)
    for i, r in enumerate(rows):
        x[i, :r.size] = r
    _assert_same(x, oracle.PER_ROW, rounding)
    # rows short enough for the kernel's in-register path
    for r in rows:
        if r.size <= 8192:
            t = np.zeros((2, (r.size + 31) // 32 * 32), np.uint16)
            t[0, :r.size] = r
            t[1, :r.size] = r[::-1]
            _assert_same(t, oracle.PER_ROW, rounding)
    # per-tensor: one scale per tensor
    for a in (0x1F7F, 0x1F80, 0x3F80):
        r = _all_magnitudes_up_to(a)
        t = np.zeros((1, (r.size + 31) // 32 * 32), np.uint16)
        t[0, :r.size] = r
        _assert_same(t.reshape(-1, 32), oracle.PER_TENSOR, rounding)


def test_zero_rows_tensor():
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    x = torch.empty((0, 64), dtype=torch.bfloat16, device=dev)
    q, s = acrl.acrl_quantize_fp8(x, acrl.SCALE_PER_TENSOR)
    torch.cuda.synchronize()
    assert float(down(s)[0]) == 1.0


N_CHUNKS = 32  # 2^32 fp32 patterns in 32 chunks of 2^27


@pytest.mark.parametrize("rounding", ROUNDINGS)
@pytest.mark.parametrize("chunk", range(N_CHUNKS))
def test_encoder_exhaustive_fp32(rounding, chunk):
    """Every one of the 2^32 fp32 bit patterns (NaNs included) encodes to the
    oracle's byte."""
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    n = (1 << 32) // N_CHUNKS
    lo = chunk * n
    bits = torch.arange(lo, lo + n, dtype=torch.int64, device=dev).to(torch.int32)
    x = bits.view(torch.float32)
    q = acrl.acrl_fp8_encode(x, rounding)
    torch.cuda.synchronize()
    xh = (np.arange(lo, lo + n, dtype=np.uint64).astype(np.uint32)).view(np.float32)
    qo = oracle.e4m3_encode(xh, rounding)
    qg = down(q)
    if not np.array_equal(qg, qo):
        i = int(np.flatnonzero(qg != qo)[0])
        raise AssertionError("pattern 0x%08x: gpu 0x%02x oracle 0x%02x"
                             % (lo + i, qg[i], qo[i]))


@pytest.mark.parametrize("operand", ["W", "H"])
@pytest.mark.parametrize("rounding", ROUNDINGS)
@pytest.mark.parametrize("name,scaling", [("q8b", oracle.PER_TENSOR), ("q17b", oracle.PER_ROW),
                                          ("mx", oracle.MX32)])
def test_full_size_lm_head_sampled_rows(name, scaling, rounding, operand):
    """Full-size W and H on the device (as the benchmark quantizes them), both
    roundings; sampled rows checked bit-exactly.  For per-tensor scaling the
    sample includes the row holding the global maximum, so the oracle derives
    the same scale."""
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    w = inputs.WORKLOADS[name]
    X = inputs.weights_bf16_torch(w, dev) if operand == "W" else inputs.hidden_bf16_torch(w, inputs.n_valid(w), dev)
    q, s = acrl.acrl_quantize_fp8(X, scaling, rounding=rounding)
    torch.cuda.synchronize()
    n = X.shape[0]
    rows = np.random.default_rng(0).choice(n, size=24, replace=False)
    rows = np.unique(np.concatenate([rows, [0, n - 1]]))
    if scaling == oracle.PER_TENSOR:
        amax_row = int(torch.argmax(X.abs().float().amax(dim=1)).item())
        rows = np.unique(np.concatenate([rows, [amax_row]]))
    idx = torch.from_numpy(rows).to(dev)
    Xb = X.index_select(0, idx).cpu().view(torch.int16).numpy().view(np.uint16)
    qo, so = oracle.quantize_fp8(Xb, scaling, rounding=rounding)
    qg = down(q.index_select(0, idx))
    assert np.array_equal(qg, qo)
    if scaling == oracle.PER_TENSOR:
        assert np.array_equal(down(s).view(np.uint8), so.view(np.uint8))
    elif scaling == oracle.PER_ROW:
        assert np.array_equal(down(s)[rows].view(np.uint8), so.view(np.uint8))
    else:
        assert np.array_equal(down(s)[rows], so)
    del X, q, s
    torch.cuda.empty_cache()


@pytest.mark.parametrize("scaling,tag", SCHEMES)
def test_row_stride(scaling, tag):
    # a column slice of a wider matrix: ld > cols (the per-tensor amax then
    # takes the per-row path instead of the flat one)
    torch, dev = torch_dev()
    from paper_2607_24062_amd import acrl
    wide = random_bf16((37, 96 + 40), 91, std=3.0)
    x = up_bf16(torch, dev, wide)[:, 8:8 + 96]
    assert not x.is_contiguous() and x.stride(0) == 136
    for rounding in ROUNDINGS:
        q, s = acrl.acrl_quantize_fp8(x, scaling, rounding)
        torch.cuda.synchronize()
        qo, so = oracle.quantize_fp8(np.ascontiguousarray(wide[:, 8:8 + 96]), scaling, rounding)
        assert np.array_equal(down(s).view(np.uint8), so.view(np.uint8))
        assert np.array_equal(down(q), qo)
