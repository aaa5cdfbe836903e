"""Pins of the oracle's quaternion algebra against scipy's Rotation and Slerp."""
import numpy as np
import pytest
from scipy.spatial.transform import Rotation, Slerp

import oracle

RNG = np.random.default_rng(11)


def _wxyz(r):
    q = r.as_quat()  # scipy: (x, y, z, w)
    return np.array([q[3], q[0], q[1], q[2]])


def _rot(q):
    return Rotation.from_quat([q[1], q[2], q[3], q[0]])


def _same_rotation(a, b, tol=1e-12):
    a = np.asarray(a) / np.linalg.norm(a)
    b = np.asarray(b) / np.linalg.norm(b)
    return min(np.abs(a - b).max(), np.abs(a + b).max()) < tol


@pytest.mark.parametrize("i", range(20))
def test_qmul_matches_composition(i):
    ra, rb = Rotation.random(2, random_state=100 + i)
    q = oracle.qmul(_wxyz(ra), _wxyz(rb))
    assert _same_rotation(q, _wxyz(ra * rb))


@pytest.mark.parametrize("i", range(20))
def test_qrot_matches_apply(i):
    r = Rotation.random(random_state=200 + i)
    v = RNG.normal(size=3)
    np.testing.assert_allclose(oracle.qrot(_wxyz(r), v), r.apply(v), atol=1e-13)


@pytest.mark.parametrize("i", range(20))
def test_rotvec_and_exp_match_scipy(i):
    r = Rotation.random(random_state=300 + i)
    q = _wxyz(r)
    if i % 2:
        q = -q  # the log map must not care about the sign
    rv = oracle.rotvec(q)
    np.testing.assert_allclose(rv, r.as_rotvec(), atol=1e-12)
    assert _same_rotation(oracle.qexp(rv), _wxyz(r))


def test_rotvec_identity_and_small_angle():
    np.testing.assert_array_equal(oracle.rotvec([1, 0, 0, 0]), [0, 0, 0])
    rv = np.array([1e-9, -2e-9, 3e-9])
    np.testing.assert_allclose(oracle.rotvec(oracle.qexp(rv)), rv, rtol=1e-9, atol=1e-20)


@pytest.mark.parametrize("i", range(20))
def test_slerp_matches_scipy(i):
    ra, rb = Rotation.random(2, random_state=400 + i)
    qa, qb = _wxyz(ra), _wxyz(rb)
    if i % 3 == 0:
        qb = -qb  # hemisphere: same rotations, same result
    sl = Slerp([0.0, 1.0], Rotation.concatenate([ra, rb]))
    for t in (0.0, 0.1, 0.37, 0.5, 0.93, 1.0):
        q = oracle.slerp(qa, qb, t)
        assert abs(np.linalg.norm(q) - 1.0) < 1e-14
        assert _same_rotation(q, _wxyz(sl([t])[0]), 1e-11)


@pytest.mark.parametrize("i", range(50))
def test_slerp_endpoints_and_constant_speed(i):
    ra, rb = Rotation.random(2, random_state=500 + i)
    qa, qb = _wxyz(ra), _wxyz(rb)
    np.testing.assert_allclose(oracle.slerp(qa, qb, 0.0), qa, atol=4e-16)
    assert _same_rotation(oracle.slerp(qa, qb, 1.0), qb, 1e-15)
    # the angle from a grows linearly in t
    ang = lambda p, q: 2 * np.arccos(min(1.0, abs(np.dot(p, q))))
    total = ang(qa, qb)
    for t in (0.25, 0.5, 0.8):
        assert abs(ang(qa, oracle.slerp(qa, qb, t)) - t * total) < 1e-7


def test_slerp_tiny_angle_and_identical():
    qa = _wxyz(Rotation.from_rotvec([0.3, -0.2, 0.1]))
    qb = oracle.qmul(qa, oracle.qexp([1e-14, 0, 0]))
    q = oracle.slerp(qa, qb, 0.5)
    assert np.all(np.isfinite(q)) and _same_rotation(q, qa, 1e-13)
    np.testing.assert_allclose(oracle.slerp(qa, qa, 0.3), qa, atol=1e-15)
