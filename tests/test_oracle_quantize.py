"""Pins of the oracle's FP8 quantizers (per-tensor, per-row, MX32), no GPU.

Checked against properties of the definitions rather than a retyped formula:
the group maximum must land on +-448, dequantized values must sit within half
an e4m3 step of the input, lossless inputs must come back unchanged, MX block
maxima must land in e4m3's top binade, and a few hand-worked MX cases.
"""
import numpy as np
import pytest

import inputs
import oracle


def _dequant_rows(q, s, scaling):
    v = oracle.e4m3_decode(q.reshape(-1)).reshape(q.shape)
    if scaling == oracle.PER_TENSOR:
        return v * float(s[0])
    if scaling == oracle.PER_ROW:
        return v * s.astype(np.float64)[:, None]
    rows, cols = q.shape
    sc = oracle.e8m0_decode(s.reshape(-1)).reshape(rows, cols // 32)
    return v * np.repeat(sc, 32, axis=1)


def _rand_bf16(rows, cols, seed, std=1.0):
    r = np.random.default_rng(seed)
    return inputs.float_to_bf16_bits((r.standard_normal((rows, cols)) * std).astype(np.float32))


@pytest.mark.parametrize("scaling", [oracle.PER_TENSOR, oracle.PER_ROW])
def test_amax_maps_to_448(scaling):
    x = _rand_bf16(7, 96, 1)
    q, s = oracle.quantize_fp8(x, scaling)
    xf = oracle.bf16_to_float(x)
    if scaling == oracle.PER_TENSOR:
        amax = np.abs(xf).max()
        assert s[0] == np.float32(amax) / np.float32(448.0)
        k = np.unravel_index(np.argmax(np.abs(xf)), xf.shape)
        assert q[k] & 0x7F == 0x7E
    else:
        amax = np.abs(xf).max(axis=1)
        assert np.array_equal(s, amax.astype(np.float32) / np.float32(448.0))
        for r in range(x.shape[0]):
            k = np.argmax(np.abs(xf[r]))
            assert q[r, k] & 0x7F == 0x7E


@pytest.mark.parametrize("scaling", [oracle.PER_TENSOR, oracle.PER_ROW, oracle.MX32])
def test_dequantized_error_within_half_step(scaling):
    x = _rand_bf16(9, 128, 2, std=3.0)
    q, s = oracle.quantize_fp8(x, scaling)
    xf = oracle.bf16_to_float(x).astype(np.float64)
    xr = _dequant_rows(q, s, scaling)
    # per element: |x - deq| <= half the e4m3 spacing at |x|/scale (3 mantissa
    # bits -> relative 2^-4), or half the subnormal step 2^-10 (times scale).
    if scaling == oracle.PER_TENSOR:
        sc = np.full_like(xf, float(s[0]))
    elif scaling == oracle.PER_ROW:
        sc = np.repeat(s.astype(np.float64)[:, None], xf.shape[1], axis=1)
    else:
        sc = np.repeat(oracle.e8m0_decode(s.reshape(-1)).reshape(s.shape), 32, axis=1)
    bound = np.maximum(np.abs(xf) * 2.0 ** -4, sc * 2.0 ** -10) * (1 + 1e-6) + 1e-30
    sat = np.abs(xf / sc) > 448  # MX may saturate a block's top values
    assert np.all((np.abs(xf - xr) <= bound) | sat)


def test_lossless_when_values_are_e4m3_and_amax_448():
    codes = np.arange(0x7F, dtype=np.uint8)
    vals = oracle.e4m3_decode(codes)
    r = np.random.default_rng(3)
    x = r.choice(np.concatenate([vals, -vals]), size=(5, 64)).astype(np.float32)
    x[:, 0] = 448.0
    xb = inputs.float_to_bf16_bits(x)
    assert np.array_equal(oracle.bf16_to_float(xb), x)  # e4m3 values are bf16-exact
    for scaling in (oracle.PER_TENSOR, oracle.PER_ROW):
        q, s = oracle.quantize_fp8(xb, scaling)
        assert np.all(s == 1.0)
        assert np.array_equal(_dequant_rows(q, s, scaling), x.astype(np.float64))


def test_zero_group_scale_is_one():
    x = np.zeros((3, 64), np.uint16)
    for scaling in (oracle.PER_TENSOR, oracle.PER_ROW):
        q, s = oracle.quantize_fp8(x, scaling)
        assert np.all(s == 1.0) and np.all(q == 0)
    q, s = oracle.quantize_fp8(x, oracle.MX32)
    assert np.all(s == 0) and np.all(q == 0)


def test_mx_hand_cases():
    # Block amax 1.0: X = 2^(0-8), code 119; the element 1.0 becomes 256 -> 0x78.
    # Block amax 3.0: X = 2^(1-8), code 120; 3.0 becomes 384 -> 0x7C.
    # Block amax 500: X = 2^(8-8) = 1, code 127; 500 saturates to 448 -> 0x7E.
    # (A "round the scale up" reading would give X = 2 and 250 -> 0x78 here.)
    rows = np.zeros((3, 32), np.float32)
    rows[0, 0] = 1.0
    rows[1, 5] = 3.0
    rows[2, 31] = 500.0
    q, s = oracle.quantize_fp8(inputs.float_to_bf16_bits(rows), oracle.MX32)
    assert list(s[:, 0]) == [119, 120, 127]
    assert q[0, 0] == 0x78 and q[1, 5] == 0x7C and q[2, 31] == 0x7E


def test_mx_block_max_lands_in_top_binade():
    x = _rand_bf16(6, 256, 4, std=10.0)
    q, s = oracle.quantize_fp8(x, oracle.MX32)
    xf = np.abs(oracle.bf16_to_float(x)).reshape(6, 8, 32)
    qb = q.reshape(6, 8, 32)
    for r in range(6):
        for b in range(8):
            k = np.argmax(xf[r, b])
            c = qb[r, b, k] & 0x7F
            # the scaled block maximum is in [256, 512): codes 0x78..0x7E (448 saturates)
            assert 0x78 <= c <= 0x7E


def test_mx_tiny_block_clamps_scale_code_at_zero():
    # amax = 2^-126 (bf16 normal) -> floor(log2) - 8 + 127 = -7 -> clamp 0
    x = np.zeros((1, 32), np.float32)
    x[0, 3] = 2.0 ** -126
    q, s = oracle.quantize_fp8(inputs.float_to_bf16_bits(x), oracle.MX32)
    assert s[0, 0] == 0
    # element = 2^-126 * 2^127 = 2 -> 0x40
    assert q[0, 3] == 0x40


def test_per_row_uses_fp32_divide():
    # an element whose fp32 quotient differs from the exact quotient must be
    # encoded from the fp32 quotient (the reading: divide in fp32, then encode)
    x = _rand_bf16(64, 64, 5)
    q, s = oracle.quantize_fp8(x, oracle.PER_ROW)
    xf = oracle.bf16_to_float(x)
    quot = (xf / s[:, None]).astype(np.float32)
    assert np.array_equal(q, oracle.e4m3_encode(quot))


def test_rejects_bad_arguments():
    with pytest.raises(ValueError):
        oracle.quantize_fp8(np.zeros((2, 33), np.uint16), oracle.MX32)
