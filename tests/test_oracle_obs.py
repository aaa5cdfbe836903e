"""Pins of the heading-frame observation."""
import numpy as np
import pytest
from scipy.spatial.transform import Rotation

import oracle
from paper_2609_09821_amd import synth

RNG = np.random.default_rng(21)


@pytest.fixture(scope="module", params=[2, 4])
def world(request):
    d = synth.make_world(request.param, n_envs=1)
    return d, oracle.World(d)


def _random_state(w, phi=0.61):
    P, Q, V, W = w.ref_state(0, np.float32(phi))
    return P, Q, V + RNG.normal(size=V.shape), W + RNG.normal(size=W.shape)


def _wxyz(r):
    q = r.as_quat()
    return np.array([q[3], q[0], q[1], q[2]])


def _rot(q):
    return Rotation.from_quat([q[1], q[2], q[3], q[0]])


@pytest.mark.parametrize("yaw", [0.0, 0.4, -2.5, np.pi])
def test_invariance_under_yaw_and_ground_translation(world, yaw):
    d, w = world
    P, Q, V, W = _random_state(w)
    o1 = w.obs(P, Q, V, W, 0.25)
    Rz = Rotation.from_euler("z", yaw)
    T = np.array([3.0, -7.0, 0.0])
    P2 = Rz.apply(P) + T
    Q2 = np.array([_wxyz(Rz * _rot(q)) for q in Q])
    o2 = w.obs(P2, Q2, Rz.apply(V), Rz.apply(W), 0.25)
    np.testing.assert_allclose(o2, o1, atol=1e-12)


def test_not_invariant_under_tilt(world):
    d, w = world
    P, Q, V, W = _random_state(w)
    Rx = Rotation.from_euler("x", 0.3)
    Q2 = np.array([_wxyz(Rx * _rot(q)) for q in Q])
    assert np.abs(w.obs(Rx.apply(P), Q2, V, W, 0.25) - w.obs(P, Q, V, W, 0.25)).max() > 1e-2


def test_root_position_and_6d_columns(world):
    d, w = world
    P, Q, V, W = _random_state(w)
    o = w.obs(P, Q, V, W, 0.5).reshape(-1)
    B = w.B
    np.testing.assert_allclose(o[0:3], [0.0, 0.0, P[0, 2]], atol=1e-15)
    for b in range(B):
        c0, c1 = o[15 * b + 3:15 * b + 6], o[15 * b + 6:15 * b + 9]
        assert abs(np.linalg.norm(c0) - 1) < 1e-12 and abs(np.linalg.norm(c1) - 1) < 1e-12
        assert abs(c0 @ c1) < 1e-12
    assert o[15 * B] == np.float32(0.5)


def test_rest_pose_closed_form(world):
    d, w = world
    B = w.B
    P = RNG.normal(size=(B, 3))
    Q = np.tile([1.0, 0, 0, 0], (B, 1))
    V, W = RNG.normal(size=(B, 3)), RNG.normal(size=(B, 3))
    o = w.obs(P, Q, V, W, 0.0).reshape(-1)
    for b in range(B):
        blk = o[15 * b:15 * b + 15]
        np.testing.assert_allclose(blk[0:3], P[b] - [P[0, 0], P[0, 1], 0], atol=1e-14)
        np.testing.assert_allclose(blk[3:9], [1, 0, 0, 0, 1, 0], atol=1e-15)
        np.testing.assert_allclose(blk[9:12], V[b], atol=1e-15)
        np.testing.assert_allclose(blk[12:15], W[b], atol=1e-15)


def test_pure_yaw_root_heading(world):
    d, w = world
    B = w.B
    psi = 0.7
    P = RNG.normal(size=(B, 3))
    Rz = Rotation.from_euler("z", psi)
    Q = np.tile(_wxyz(Rz), (B, 1))
    V = np.tile([1.0, 0.0, 0.0], (B, 1))
    o = w.obs(P, Q, V, V, 0.0).reshape(-1)
    # in the heading frame the root is unrotated and a world +x velocity reads
    # (cos psi, -sin psi, 0)
    np.testing.assert_allclose(o[3:9], [1, 0, 0, 0, 1, 0], atol=1e-15)
    np.testing.assert_allclose(o[9:12], [np.cos(psi), -np.sin(psi), 0], atol=1e-15)


def test_degenerate_heading_is_identity(world):
    d, w = world
    B = w.B
    P, Q, V, W = _random_state(w)
    Q = Q.copy()
    Q[0] = _wxyz(Rotation.from_euler("y", -np.pi / 2))  # forward axis points straight up
    o = w.obs(P, Q, V, W, 0.0).reshape(-1)
    np.testing.assert_allclose(o[15 * 1:15 * 1 + 3], P[1] - [P[0, 0], P[0, 1], 0], atol=1e-14)
