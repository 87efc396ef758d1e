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
