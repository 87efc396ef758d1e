"""Pins of the oracle's FP8 e4m3 / e8m0 formats (no GPU).

The oracle encodes with exponent/mantissa arithmetic.  These tests check it
against things that do not share that arithmetic: the OCP hand values in
tests/golden/, a brute-force search over all 254 finite codes, and torch's own
float8_e4m3fn conversion (a library routine) on its non-saturating range.
"""
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _finite_codes():
    codes = np.arange(256, dtype=np.uint8)
    vals = oracle.e4m3_decode(codes)
    keep = ~np.isnan(vals)
    return codes[keep], vals[keep]


def test_hand_values():
    rows = []
    with open(os.path.join(GOLDEN, "e4m3_hand_values.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                v, c = line.split()[:2]
                rows.append((float(v), int(c, 16)))
    x = np.array([r[0] for r in rows], np.float32)
    got = oracle.e4m3_encode(x)
    assert [hex(g) for g in got] == [hex(r[1]) for r in rows]


def test_decode_table_properties():
    codes, vals = _finite_codes()
    assert len(codes) == 254            # 0x7F and 0xFF are the NaNs
    assert vals.max() == 448.0 and vals.min() == -448.0
    pos = np.sort(vals[vals > 0])
    assert pos[0] == 2.0 ** -9          # smallest subnormal
    assert np.all(np.diff(pos) > 0)
    # positive codes 0x00..0x7E are monotone in value
    assert np.all(np.diff(oracle.e4m3_decode(np.arange(0x7F, dtype=np.uint8))) > 0)
    assert np.isnan(oracle.e4m3_decode(np.array([0x7F, 0xFF], np.uint8))).all()


@pytest.mark.parametrize("rounding", [oracle.ROUND_NEAREST_EVEN, oracle.ROUND_TOWARD_ZERO])
def test_every_code_round_trips(rounding):
    codes, vals = _finite_codes()
    got = oracle.e4m3_encode(vals.astype(np.float32), rounding)
    assert np.array_equal(got, codes)


def _brute_nearest(x: np.ndarray) -> np.ndarray:
    """Nearest finite e4m3 by exhaustive search; ties to the even code;
    magnitudes past 448 saturate; NaN -> 0x7F|sign."""
    codes, vals = _finite_codes()
    pos = codes[(vals > 0) | ((vals == 0) & (codes == 0))]
    pv = oracle.e4m3_decode(pos)
    order = np.argsort(pv)
    pos, pv = pos[order], pv[order]
    a = np.abs(x.astype(np.float64))
    dist = np.abs(a[:, None] - pv[None, :])
    best = dist.min(axis=1, keepdims=True)
    cand = dist == best
    n_cand = cand.sum(axis=1)
    pick = np.where(n_cand == 1, pos[np.argmax(cand, axis=1)], 0)
    tie = n_cand == 2
    if tie.any():
        idx = np.argwhere(cand[tie])
        first = pos[idx[0::2, 1]]
        second = pos[idx[1::2, 1]]
        pick[tie] = np.where(first % 2 == 0, first, second)
    pick = np.where(a >= 448.0, 0x7E, pick)
    sign = (np.signbit(x)).astype(np.uint8) << 7
    out = (pick.astype(np.uint8) | sign)
    out = np.where(np.isnan(x), 0x7F | sign, out)
    return out.astype(np.uint8)


def _brute_toward_zero(x: np.ndarray) -> np.ndarray:
    codes, vals = _finite_codes()
    pos = codes[(vals > 0) | ((vals == 0) & (codes == 0))]
    pv = oracle.e4m3_decode(pos)
    order = np.argsort(pv)
    pos, pv = pos[order], pv[order]
    a = np.abs(x.astype(np.float64))
    k = np.searchsorted(pv, a, side="right") - 1   # largest value <= a
    pick = pos[np.clip(k, 0, len(pos) - 1)]
    sign = (np.signbit(x)).astype(np.uint8) << 7
    return (pick.astype(np.uint8) | sign).astype(np.uint8)


def _bf16_all_finite():
    b = np.arange(65536, dtype=np.uint32)
    f = (b << 16).view(np.float32)
    return f[np.isfinite(f)]


def _random_fp32(n, seed):
    r = np.random.default_rng(seed)
    # log-uniform magnitudes over the whole e4m3 range and beyond, both signs
    mag = np.exp2(r.uniform(-14, 10, size=n)).astype(np.float32)
    x = mag * np.where(r.random(n) < 0.5, -1, 1).astype(np.float32)
    # plus exact midpoints between adjacent codes
    codes, vals = _finite_codes()
    pv = np.sort(np.unique(np.abs(vals)))
    mids = ((pv[1:] + pv[:-1]) / 2).astype(np.float32)
    return np.concatenate([x, mids, -mids, np.nextafter(mids, np.float32(0)),
                           np.nextafter(mids, np.float32(1e9))])


def test_nearest_matches_brute_force_on_all_bf16():
    x = _bf16_all_finite()
    assert np.array_equal(oracle.e4m3_encode(x), _brute_nearest(x))


def test_nearest_matches_brute_force_on_random_fp32():
    x = _random_fp32(200_000, 7)
    assert np.array_equal(oracle.e4m3_encode(x), _brute_nearest(x))


def test_toward_zero_matches_brute_force():
    x = np.concatenate([_bf16_all_finite(), _random_fp32(100_000, 8)])
    got = oracle.e4m3_encode(x, oracle.ROUND_TOWARD_ZERO)
    assert np.array_equal(got, _brute_toward_zero(x))


def test_specials():
    x = np.array([np.inf, -np.inf, np.nan, -np.nan, 1e30, -1e30], np.float32)
    got = oracle.e4m3_encode(x)
    assert got[0] == 0x7E and got[1] == 0xFE
    assert got[2] & 0x7F == 0x7F and got[3] & 0x7F == 0x7F
    assert got[4] == 0x7E and got[5] == 0xFE


def test_matches_torch_float8_e4m3fn_inside_range():
    torch = pytest.importorskip("torch")
    x = np.concatenate([_bf16_all_finite(), _random_fp32(100_000, 9)])
    x = x[np.abs(x) <= 448.0]
    want = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(oracle.e4m3_encode(x), want)


def test_e8m0_decode():
    c = np.array([0, 1, 119, 120, 127, 128, 254, 255], np.uint8)
    v = oracle.e8m0_decode(c)
    assert v[0] == 2.0 ** -127 and v[1] == 2.0 ** -126
    assert v[2] == 2.0 ** -8 and v[3] == 2.0 ** -7
    assert v[4] == 1.0 and v[5] == 2.0 and v[6] == 2.0 ** 127
    assert np.isnan(v[7])
