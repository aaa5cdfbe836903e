"""Pins of the oracle's random numbers: Philox4x32-10 and the normal draws."""
import os

import numpy as np
import pytest
from scipy import stats

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.txt")


def _kat():
    rows = []
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        v = [int(x, 16) for x in line.split()]
        rows.append((v[0:4], v[4:6], v[6:10]))
    return rows


@pytest.mark.parametrize("ctr,key,expect", _kat())
def test_philox_known_answers(ctr, key, expect):
    assert list(oracle.philox(ctr, key)) == expect


def test_philox_counter_sensitivity():
    a = oracle.philox([1, 2, 3, 4], [5, 6])
    for i in range(4):
        c = [1, 2, 3, 4]
        c[i] ^= 1
        assert not np.array_equal(oracle.philox(c, [5, 6]), a)


def test_normals_distribution():
    seed = 0x1234_5678_9ABC_DEF0
    z = np.concatenate([oracle.normals(seed, e, 7, 0, 3) for e in range(6000)])
    assert abs(z.mean()) < 0.03
    assert abs(z.var() - 1.0) < 0.04
    assert stats.kstest(z, "norm").pvalue > 1e-3
    # pairs from one Box-Muller draw are uncorrelated
    zz = z.reshape(-1, 4)
    assert abs(np.corrcoef(zz[:, 0], zz[:, 1])[0, 1]) < 0.04


def test_normals_extreme_words_finite():
    # the uniform map excludes 0 and 1, so every word gives a finite normal
    for e in range(64):
        z = oracle.normals(0, e, 0xFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF)
        assert np.all(np.isfinite(z))


def test_box_muller_worked_example():
    # A hand-worked draw.  The first published known-answer vector (counter 0,
    # key 0) is the action-noise block (env 0, step counter 0, block 0, tag 0)
    # under seed 0.  Each word x maps to the open-interval uniform
    # (2 (x >> 9) + 1) 2^-24, done here by hand:
    #   x0 = 0x6627e8d5 = 1713891541, x0 >> 9 = 3347444 (rest 213): u0 =  6694889 / 2^24
    #   x1 = 0xe169c58d = 3781805453, x1 >> 9 = 7386338 (rest 397): v0 = 14772677 / 2^24
    #   x2 = 0xbc57ac4c = 3159862348, x2 >> 9 = 6171606 (rest  76): u1 = 12343213 / 2^24
    #   x3 = 0x9b00dbd8 = 2600524760, x3 >> 9 = 5079149 (rest 472): v1 = 10158299 / 2^24
    # and the pairs (u0, v0), (u1, v1) give z = sqrt(-2 ln u) (cos 2 pi v, sin 2 pi v),
    # evaluated at 40 digits.  Swapping u and v, cos and sin, or the two word
    # pairs changes every one of the four values.
    import mpmath
    words = [0x6627e8d5, 0xe169c58d, 0xbc57ac4c, 0x9b00dbd8]
    assert list(oracle.philox([0, 0, 0, 0], [0, 0])) == words
    hand = [(1713891541, 3347444, 213, 6694889), (3781805453, 7386338, 397, 14772677),
            (3159862348, 6171606, 76, 12343213), (2600524760, 5079149, 472, 10158299)]
    for x, (dec, q, rest, odd) in zip(words, hand):
        assert x == dec == 512 * q + rest and 0 <= rest < 512 and odd == 2 * q + 1
    mpmath.mp.dps = 40
    z = []
    for u_num, v_num in ((hand[0][3], hand[1][3]), (hand[2][3], hand[3][3])):
        u, v = mpmath.mpf(u_num) / 2 ** 24, mpmath.mpf(v_num) / 2 ** 24
        r = mpmath.sqrt(-2 * mpmath.log(u))
        z += [r * mpmath.cos(2 * mpmath.pi * v), r * mpmath.sin(2 * mpmath.pi * v)]
    got = oracle.normals(0, 0, 0, 0, 0)
    for g, e in zip(got, z):
        assert abs(g - float(e)) <= 1e-13 * max(1.0, abs(float(e))), (g, e)
