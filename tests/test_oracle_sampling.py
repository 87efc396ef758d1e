"""Pins of the oracle's Gumbel-max sampler from mu (no GPU).

The counter-based generator is Philox4x32-10, checked against its published
known-answer vectors (tests/golden/philox4x32_10_kat.txt).  The sampler is
checked against what the Gumbel-max trick guarantees: a draw from
softmax(z) (frequencies over many independent tokens), invariance to a
constant shift of the logits, and a dominant logit always winning.
"""
import math
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _kat():
    rows = []
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                rows.append([int(x, 16) for x in line.split()])
    return rows


@pytest.mark.parametrize("row", _kat())
def test_philox_known_answers(row):
    got = oracle.philox4x32_10(row[0:4], row[4:6])
    assert [int(x) for x in got] == row[6:10]


def test_uniform_range_and_mean():
    u = np.array([oracle.sample_uniform(7, t, v) for t in range(40) for v in range(50)])
    assert (u > 0).all() and (u < 1).all()
    assert abs(u.mean() - 0.5) < 4 * math.sqrt(1 / 12 / u.size)
    # the four words of one Philox call serve v = 4m .. 4m+3
    w = oracle.philox4x32_10([3, 11, 0, 0], [7, 0])
    for i in range(4):
        assert oracle.sample_uniform(7, 11, 12 + i) == ((int(w[i]) >> 9) + 0.5) / 2 ** 23


def test_gumbel_max_draws_from_the_softmax():
    z = np.array([0.0, 1.0, -0.5, 2.0, 0.3])
    p = np.exp(z - z.max())
    p /= p.sum()
    n = 20000
    ids, _ = oracle.gumbel_sample(np.tile(z, (n, 1)), seed=123)
    freq = np.bincount(ids, minlength=z.size) / n
    sigma = np.sqrt(p * (1 - p) / n)
    assert (np.abs(freq - p) < 5 * sigma).all(), (freq, p)


def test_gumbel_shift_invariance_and_dominant_logit():
    r = np.random.default_rng(5)
    z = r.normal(size=(64, 37))
    a, ka = oracle.gumbel_sample(z, seed=9, row_offset=1000)
    b, kb = oracle.gumbel_sample(z + 3.25, seed=9, row_offset=1000)
    assert np.array_equal(a, b)
    np.testing.assert_allclose(kb - ka, 3.25, rtol=0, atol=1e-12)
    z2 = z.copy()
    z2[np.arange(64), 17] = 60.0
    c, _ = oracle.gumbel_sample(z2, seed=9, row_offset=1000)
    assert (c == 17).all()
    # a different seed or token offset gives a different stream
    d, _ = oracle.gumbel_sample(z, seed=10, row_offset=1000)
    e, _ = oracle.gumbel_sample(z, seed=9, row_offset=0)
    assert not np.array_equal(a, d) and not np.array_equal(a, e)


# ------------------------------------------------------------ blockwise Gumbel-max
# The draw the mu kernel makes: one Gumbel key per block of 16 vocabulary
# rows plus an inverse-CDF pick inside the winning block.  Pinned by what
# makes it a draw from softmax(z): row and block frequencies over many
# independent tokens, a single block reducing to the inverse CDF with the
# documented uniform, shift invariance, a dominant logit.

def _block_rows(k, V):
    return [v for q in range(4) for j in range(4)
            for v in [32 * (k // 2) + 8 * q + 4 * (k % 2) + j] if v < V]


def test_block_partition_covers_the_vocabulary():
    for V in (1, 4, 5, 31, 32, 33, 70, 151936 // 64):
        rows = sorted(v for k in range(2 * ((V + 31) // 32)) for v in _block_rows(k, V))
        assert rows == list(range(V))
        assert all(oracle.block_of_row(v) == k for k in range(2 * ((V + 31) // 32)) for v in _block_rows(k, V))


@pytest.mark.parametrize("V", [70, 37])
def test_block_gumbel_draws_from_the_softmax(V):
    r = np.random.default_rng(V)
    z = r.normal(0, 1.5, size=V)
    z[3] += 2.0
    p = np.exp(z - z.max())
    p /= p.sum()
    n = 40000
    ids, keys, blocks = oracle.block_gumbel_sample(np.tile(z, (n, 1)), seed=77, row_offset=5)
    assert np.array_equal(oracle.block_of_row(ids), blocks)
    freq = np.bincount(ids, minlength=V) / n
    sigma = np.sqrt(p * (1 - p) / n)
    assert (np.abs(freq - p) < 5 * sigma + 2.0 / n).all()  # + two draws for rows of tiny p
    chi2 = float(((freq - p) ** 2 / p).sum() * n)
    assert chi2 < V + 6 * math.sqrt(2 * V)  # chi-square with V - 1 degrees of freedom
    # the winning block's frequency is its total probability
    pb = np.bincount(oracle.block_of_row(np.arange(V)), weights=p)
    fb = np.bincount(blocks, minlength=pb.size) / n
    assert (np.abs(fb - pb) < 5 * np.sqrt(pb * (1 - pb) / n) + 1e-12).all()


def test_single_block_is_the_inverse_cdf_of_its_second_uniform():
    # V <= 4: one block (rows 0..3); its pick uses u' = word 1 of Philox on
    # counter (0, t, 0, 0) (k = 0: floor(v/64) = 0, k mod 2 = 0, e = 0)
    r = np.random.default_rng(3)
    n, V, seed = 300, 4, 0x1234_5678_9ABC
    z = r.normal(size=(n, V))
    ids, _, blocks = oracle.block_gumbel_sample(z, seed=seed, row_offset=11)
    assert (blocks == 0).all()
    u = np.array([((int(oracle.philox4x32_10([0, 11 + t, 0, 0], [seed & 0xFFFFFFFF, seed >> 32])[1]) >> 9) + 0.5)
                  / 2 ** 23 for t in range(n)])
    assert np.array_equal(ids, oracle.sample_inverse_cdf(z, u))


def test_block_gumbel_shift_invariance_dominant_logit_and_offsets():
    r = np.random.default_rng(8)
    z = r.normal(size=(64, 300))
    a, ka, ba = oracle.block_gumbel_sample(z, seed=9, row_offset=1000)
    b, kb, bb = oracle.block_gumbel_sample(z + 3.25, seed=9, row_offset=1000)
    assert np.array_equal(a, b) and np.array_equal(ba, bb)
    np.testing.assert_allclose(kb - ka, 3.25, rtol=0, atol=1e-12)
    z2 = z.copy()
    z2[:, 217] = 60.0
    c, _, _ = oracle.block_gumbel_sample(z2, seed=9, row_offset=1000)
    assert (c == 217).all()
    # rows drawn in two calls with their offsets = one call
    d1, _, _ = oracle.block_gumbel_sample(z[:20], seed=9, row_offset=1000)
    d2, _, _ = oracle.block_gumbel_sample(z[20:], seed=9, row_offset=1020)
    assert np.array_equal(np.concatenate([d1, d2]), a)
    e, _, _ = oracle.block_gumbel_sample(z, seed=10, row_offset=1000)
    assert not np.array_equal(a, e)
