"""Pins of reference sampling and forward kinematics (positions and velocities)."""
import numpy as np
import pytest
from scipy.spatial.transform import Rotation

import oracle
from paper_2609_09821_amd import synth
from tests.worlds import clip_from_arrays, custom_world, rest_offsets_world


def _same_rot(a, b, tol):
    return min(np.abs(a - b).max(), np.abs(a + b).max()) < tol


@pytest.mark.parametrize("cfg", [2, 4])
def test_identity_pose_gives_rest_skeleton(cfg):
    d = synth.make_world(cfg, n_envs=1)
    w = oracle.World(d)
    B = w.B
    ident = np.tile([1.0, 0, 0, 0], (B, 1))
    P, Q, V, W = w.fk(np.zeros(3), [1, 0, 0, 0], np.zeros(3), np.zeros(3), ident,
                      np.zeros((B, 3)))
    np.testing.assert_allclose(P, rest_offsets_world(d), atol=1e-15)
    np.testing.assert_array_equal(Q, ident)
    np.testing.assert_array_equal(V, 0)
    np.testing.assert_array_equal(W, 0)


@pytest.mark.parametrize("th", [(0.3, 0.7, -1.1), (-2.0, 1.0, 0.25), (0.0, 0.0, 0.0)])
def test_planar_chain_closed_form(th):
    # three bodies in a chain, every link along local +x, rotations about z
    L1, L2 = 0.4, 0.3
    d = custom_world([-1, 0, 1], [0, 1, 1], [[0, 0, 0], [L1, 0, 0], [L2, 0, 0]], [1, 1, 1],
                     [clip_from_arrays(np.zeros((2, 3)), np.tile([1, 0, 0, 0], (2, 1)),
                                       np.tile([1, 0, 0, 0], (2, 2, 1)))])
    w = oracle.World(d)
    rz = lambda a: np.array([np.cos(a / 2), 0, 0, np.sin(a / 2)])
    ql = np.array([[1, 0, 0, 0], rz(th[1]), rz(th[2])], float)
    wz = np.array([0.0, 0.5, -0.25])  # joint rates about z
    wl = np.array([[0, 0, 0], [0, 0, wz[1]], [0, 0, wz[2]]])
    P, Q, V, W = w.fk([1.0, 2.0, 0.5], rz(th[0]), [0, 0, 0], [0, 0, wz[0]], ql, wl)
    a0, a1 = th[0], th[0] + th[1]
    p1 = np.array([1.0 + L1 * np.cos(a0), 2.0 + L1 * np.sin(a0), 0.5])
    p2 = p1 + [L2 * np.cos(a1), L2 * np.sin(a1), 0]
    np.testing.assert_allclose(P[1], p1, atol=1e-15)
    np.testing.assert_allclose(P[2], p2, atol=1e-15)
    assert _same_rot(Q[2], rz(th[0] + th[1] + th[2]), 1e-15)
    # planar angular rates add; body 2's origin moves with the rates of body 0 and 1
    np.testing.assert_allclose(W[2], [0, 0, wz[0] + wz[1] + wz[2]], atol=1e-15)
    v1 = wz[0] * L1 * np.array([-np.sin(a0), np.cos(a0), 0])
    v2 = v1 + (wz[0] + wz[1]) * L2 * np.array([-np.sin(a1), np.cos(a1), 0])
    np.testing.assert_allclose(V[1], v1, atol=1e-15)
    np.testing.assert_allclose(V[2], v2, atol=1e-15)


def _phase_grid(F):
    # phases on a 2^-12 grid inside segment interiors: phi * (F-1) and
    # (phi +- 2^-15) * (F-1) are then exact in fp32 (at most 24 significant bits)
    out = []
    for i in range(0, F - 1, max(1, (F - 1) // 7)):
        out.append(np.float32(np.round((i + 0.5) / (F - 1) * 4096) / 4096))
    return out


@pytest.mark.parametrize("cfg", [2, 4])
def test_reference_velocities_are_time_derivatives(cfg):
    d = synth.make_world(cfg, n_envs=1)
    w = oracle.World(d)
    F = d["clips"][0]["n_frames"]
    fps = d["clips"][0]["fps"]
    h = np.float32(2.0 ** -15)
    for phi in _phase_grid(F):
        pp, pm = np.float32(phi + h), np.float32(phi - h)
        i_p, a_p = oracle.phase_index(F, pp)
        i_m, a_m = oracle.phase_index(F, pm)
        assert i_p == i_m  # both inside one segment
        _, a0 = oracle.phase_index(F, phi)
        assert float(a_p) - float(a0) == float(a0) - float(a_m)  # centred difference
        Pp, Qp, _, _ = w.ref_state(0, pp)
        Pm, Qm, _, _ = w.ref_state(0, pm)
        _, _, V0, W0 = w.ref_state(0, phi)
        # the blend advances by one per frame, i.e. at fps per second
        dt = (float(a_p) - float(a_m)) / fps
        V_fd = (Pp - Pm) / dt
        np.testing.assert_allclose(V0, V_fd, atol=1e-6 * (1 + np.abs(V0).max()))
        for b in range(w.B):
            rel = Rotation.from_quat(np.r_[Qp[b][1:], Qp[b][0]]) * \
                Rotation.from_quat(np.r_[Qm[b][1:], Qm[b][0]]).inv()
            W_fd = rel.as_rotvec() / dt
            np.testing.assert_allclose(W0[b], W_fd, atol=1e-6 * (1 + np.abs(W0[b]).max()))


@pytest.mark.parametrize("cfg", [2, 3, 5])
def test_reference_hits_clip_frames(cfg):
    d = synth.make_world(cfg, n_envs=1)
    w = oracle.World(d)
    for k, c in enumerate(d["clips"]):
        F = c["n_frames"]
        for i in (0, 1, F // 2, F - 2, F - 1):
            phi = np.float32(i / (F - 1))
            i0, a = oracle.phase_index(F, phi)
            if np.float32(phi * np.float32(F - 1)) != np.float32(i):
                continue  # phase not exactly on the frame in fp32
            P, Q, V, W = w.ref_state(k, phi)
            np.testing.assert_allclose(P[0], c["root_pos"][i], atol=1e-12)
            assert _same_rot(Q[0], c["root_quat"][i].astype(np.float64)
                             / np.linalg.norm(c["root_quat"][i].astype(np.float64)), 1e-7)


@pytest.mark.parametrize("F", [2, 3, 30, 120, 300])
def test_phase_index_brute_force(F):
    phis = [0.0, 1.0, np.nextafter(np.float32(1), np.float32(0)), 1e-30, 0.5]
    phis += [np.float32(i / (F - 1)) for i in range(F)]
    phis += list(np.random.default_rng(F).random(2000).astype(np.float32))
    for phi in phis:
        phi = np.float32(phi)
        i0, a = oracle.phase_index(F, phi)
        s = np.float32(phi * np.float32(F - 1))
        assert 0 <= i0 <= F - 2
        assert np.float32(0) <= a <= np.float32(1)
        assert np.float32(np.float32(i0) + a) == s  # decomposition is exact
        if s < F - 1:
            assert i0 == int(np.floor(s))
        else:
            assert i0 == F - 2 and a == 1


def test_dphi_definition():
    d = synth.make_world(3, n_envs=1)
    w = oracle.World(d)
    for k, c in enumerate(d["clips"]):
        exp = np.float32((1.0 / 30.0) * np.float64(np.float32(c["fps"])) / (c["n_frames"] - 1))
        assert w.dphi(k) == exp
