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
