"""Pins of the training-step terms: the multiplicative five-term reward and
the observation extras (future reference frames of the root and end
effectors, previous action).  Closed forms are derived by hand from a
perturbed reference pose; the heading-frame encoding is recomputed with
numpy."""
import numpy as np
import pytest
from scipy.spatial.transform import Rotation

import oracle
from paper_2609_09821_amd import synth

RNG = np.random.default_rng(11)


def _world(cfg=6, n=1, **over):
    d = synth.make_world(cfg, n_envs=n, **over)
    return d, oracle.World(d)


def _R(q):
    return Rotation.from_quat([q[1], q[2], q[3], q[0]]).as_matrix()


def _qmul(a, b):
    w1, x1, y1, z1 = a
    w2, x2, y2, z2 = b
    return np.array([w1 * w2 - x1 * x2 - y1 * y2 - z1 * z2, w1 * x2 + x1 * w2 + y1 * z2 - z1 * y2,
                     w1 * y2 - x1 * z2 + y1 * w2 + z1 * x2, w1 * z2 + x1 * y2 - y1 * x2 + z1 * w2])


def _conj(q):
    return np.array([q[0], -q[1], -q[2], -q[3]])


def _qexp(r):
    x = Rotation.from_rotvec(r).as_quat()
    return np.array([x[3], x[0], x[1], x[2]])


def _local_pose(d, w, k, phi):
    """The reference at (k, phi) as root state + joint rotations and joint
    angular velocities (parent frame), derived from its world state."""
    P, Q, V, W = w.ref_state(k, phi)
    par = d["skeleton"]["parent"]
    ql = np.zeros((w.B, 4))
    wl = np.zeros((w.B, 3))
    ql[0] = [1, 0, 0, 0]
    for b in range(1, w.B):
        p = par[b]
        ql[b] = _qmul(_conj(Q[p]), Q[b])
        wl[b] = _R(Q[p]).T @ (W[b] - W[p])
    return P, Q, V, W, ql, wl


def _leaves(d):
    par = d["skeleton"]["parent"]
    return [b for b in range(len(par)) if b not in set(par[1:])]


def _subtree(d, b):
    par = d["skeleton"]["parent"]
    out = {b}
    for c in range(b + 1, len(par)):
        if par[c] in out:
            out.add(c)
    return out


def test_obs_dim_formula():
    d, w = _world()
    n_ee = len(_leaves(d))
    assert n_ee == 5
    assert w.D == 15 * 24 + 1 + 2 * (1 + n_ee) * 9 + 69 == 538
    assert w.D == synth.obs_dim(24, n_ee, 69, d["config"]) == d["policy"]["dims"][0]


@pytest.mark.parametrize("phi", [0.0, 0.3711, 0.9])
def test_reference_itself_has_zero_error(phi):
    d, w = _world()
    P, Q, V, W = w.ref_state(0, phi)
    m = w.mreward(P, Q, W, 0, phi)
    for key in ("e_jrot", "e_jvel", "e_com", "e_eepos", "e_eerot"):
        assert m[key] < 1e-20, (key, m[key])
    assert m["r"] == pytest.approx(1.0, abs=1e-12)


def test_one_joint_rotated():
    d, w = _world()
    phi = 0.42
    P, Q, V, W, ql, wl = _local_pose(d, w, 0, phi)
    leaves = set(_leaves(d))
    cfg = d["config"]
    for b in (1, 3, 7, 12, 20):
        for th in (0.05, 0.4, 1.3):
            axis = RNG.normal(size=3)
            axis /= np.linalg.norm(axis)
            q2 = ql.copy()
            q2[b] = _qmul(ql[b], _qexp(th * axis))
            Ps, Qs, Vs, Ws = w.fk(P[0], Q[0], V[0], W[0], q2, wl)
            m = w.mreward(Ps, Qs, Ws, 0, phi)
            n_ee = len(_subtree(d, b) & leaves)
            assert m["e_jrot"] == pytest.approx(th * th, rel=1e-9)
            assert m["e_eerot"] == pytest.approx(n_ee * th * th, rel=1e-9)
            assert m["e_jvel"] < 1e-20
            expect = np.exp(-cfg["m_jrot"] * th * th) * np.exp(-cfg["m_eerot"] * n_ee * th * th) \
                * np.exp(-cfg["m_com"] * m["e_com"]) * np.exp(-cfg["m_eepos"] * m["e_eepos"])
            assert m["r"] == pytest.approx(expect, rel=1e-12)


def test_root_rotated():
    d, w = _world()
    phi = 0.6
    P, Q, V, W, ql, wl = _local_pose(d, w, 0, phi)
    th = 0.3
    Q0 = _qmul(Q[0], _qexp(th * np.array([0.0, 0.6, 0.8])))
    Ps, Qs, Vs, Ws = w.fk(P[0], Q0, V[0], W[0], ql, wl)
    m = w.mreward(Ps, Qs, Ws, 0, phi)
    assert m["e_jrot"] == pytest.approx(th * th, rel=1e-9)
    assert m["e_eerot"] == pytest.approx(len(_leaves(d)) * th * th, rel=1e-9)
    assert m["e_jvel"] < 1e-20


def test_one_joint_velocity_changed():
    d, w = _world()
    phi = 0.2
    P, Q, V, W, ql, wl = _local_pose(d, w, 0, phi)
    for b in (2, 9, 23):
        dv = RNG.normal(size=3) * 0.7
        w2 = wl.copy()
        w2[b] = wl[b] + dv
        Ps, Qs, Vs, Ws = w.fk(P[0], Q[0], V[0], W[0], ql, w2)
        m = w.mreward(Ps, Qs, Ws, 0, phi)
        assert m["e_jvel"] == pytest.approx(float(dv @ dv), rel=1e-9)
        assert m["e_jrot"] < 1e-20 and m["e_eerot"] < 1e-20
        assert m["e_eepos"] < 1e-20 and m["e_com"] < 1e-20


def test_rigid_translation():
    d, w = _world()
    phi = 0.77
    P, Q, V, W = w.ref_state(0, phi)
    sh = np.array([0.02, -0.05, 0.01])
    m = w.mreward(P + sh, Q, W, 0, phi)
    x = float(sh @ sh)
    assert m["e_com"] == pytest.approx(x, rel=1e-9)
    assert m["e_eepos"] == pytest.approx(len(_leaves(d)) * x, rel=1e-9)
    assert m["e_jrot"] < 1e-20 and m["e_jvel"] < 1e-20 and m["e_eerot"] < 1e-20
    cfg = d["config"]
    assert m["r"] == pytest.approx(np.exp(-cfg["m_com"] * x) * np.exp(-cfg["m_eepos"] * 5 * x),
                                   rel=1e-12)


def test_multiplicative_form_drives_the_step():
    # the step's reward is the multiplicative one for this workload
    d, w = _world(n=40)
    st = w.state(40)
    w.reset_envs(st)
    w.standin(st, d["sigma_joint"], d["sigma_vel"])
    sim = st.copy()
    phases = []
    for e in range(40):
        phi1 = np.float32(st.phase[e] + w.dphi(st.clip[e]))
        phases.append(min(phi1, np.float32(1.0)))
    w.env_step(st, prev_action=np.zeros((40, w.A), np.float32))
    for e in range(40):
        P = sim.pos[:, :, e].astype(np.float64)
        Q = sim.quat[:, :, e].astype(np.float64)
        W = sim.angvel[:, :, e].astype(np.float64)
        m = w.mreward(P, Q, W, int(sim.clip[e]), phases[e])
        assert st.reward[e] == np.float32(m["r"])


def _heading(q0, p0):
    R0 = _R(q0)
    fx, fy = R0[0, 0], R0[1, 0]
    n = np.hypot(fx, fy)
    c, s = (1.0, 0.0) if n * n < 1e-12 else (fx / n, fy / n)
    HT = np.array([[c, s, 0], [-s, c, 0], [0, 0, 1.0]])
    return HT, np.array([p0[0], p0[1], 0.0])


def _frame9(HT, org, P, Q):
    M = HT @ _R(Q)
    return np.concatenate([HT @ (P - org), M[:, 0], M[:, 1]])


@pytest.mark.parametrize("cfg", [6])
def test_future_frames_and_previous_action(cfg):
    N = 30
    d, w = _world(cfg, n=N)
    st = w.state(N)
    st.n[:] = np.arange(N, dtype=np.uint32) * 5
    w.reset_envs(st)
    for _ in range(3):
        w.standin(st, d["sigma_joint"], d["sigma_vel"])
        w.env_step(st, prev_action=np.zeros((N, w.A), np.float32))
    w.standin(st, d["sigma_joint"], d["sigma_vel"])
    prev = RNG.normal(size=(N, w.A)).astype(np.float32)
    w.env_step(st, prev_action=prev)
    leaves = _leaves(d)
    D0 = 15 * w.B + 1
    K = d["config"]["obs_future"]
    for e in range(N):
        k = int(st.clip[e])
        HT, org = _heading(st.quat[0, :, e].astype(np.float64), st.pos[0, :, e].astype(np.float64))
        ph = np.float32(st.phase[e])
        o = st.obs[:, e].astype(np.float64)
        idx = D0
        for j in range(K):
            ph = np.float32(ph + w.dphi(k))
            P, Q, V, W = w.ref_state(k, min(ph, np.float32(1.0)))
            for b in [0] + leaves:
                np.testing.assert_allclose(o[idx:idx + 9], _frame9(HT, org, P[b], Q[b]),
                                           atol=2e-6, rtol=0)
                idx += 9
        done = st.terminated[e] or st.truncated[e]
        expect = np.zeros(w.A, np.float32) if done else prev[e]
        np.testing.assert_array_equal(st.obs[idx:idx + w.A, e], expect)
        assert idx + w.A == w.D


def test_static_clip_future_frames_equal_current_rows():
    # a clip whose frames are all equal: every future reference frame is the
    # current reference, so a freshly reset env's future blocks repeat the
    # position and 6D rows of the root and the end effectors
    d = synth.make_world(6, n_envs=8)
    c = d["clips"][0]
    for key in ("root_pos", "root_quat", "local_quat"):
        c[key] = np.repeat(c[key][:1], c["n_frames"], axis=0)
    w = oracle.World(d)
    st = w.state(8)
    w.reset_envs(st)
    D0 = 15 * w.B + 1
    leaves = _leaves(d)
    for e in range(8):
        idx = D0
        for j in range(d["config"]["obs_future"]):
            for b in [0] + leaves:
                np.testing.assert_allclose(st.obs[idx:idx + 9, e], st.obs[15 * b:15 * b + 9, e],
                                           atol=1e-6)
                idx += 9
        assert np.all(st.obs[idx:, e] == 0.0)          # no previous action after a reset


def test_quaternion_sign_does_not_matter():
    # q and -q are the same rotation: negating stored orientations leaves every
    # rotation error at zero
    d, w = _world()
    phi = 0.33
    P, Q, V, W = w.ref_state(0, phi)
    Qn = Q.copy()
    Qn[::2] *= -1.0
    m = w.mreward(P, Qn, W, 0, phi)
    assert m["e_jrot"] < 1e-20 and m["e_eerot"] < 1e-20
    assert m["r"] == pytest.approx(1.0, abs=1e-12)


def test_future_frames_hold_the_clip_end():
    # envs whose next phases pass the end of the clip (without truncating this
    # step) see the last reference frame repeated
    N = 16
    d, w = _world(n=N)
    st = w.state(N)
    w.reset_envs(st)
    dphi = w.dphi(0)
    st.clip[:] = 0
    st.t[:] = 10
    # after the step the phase lies in [1 - dphi, 1): not truncated, future phases >= 1
    st.phase[:] = np.float32(1.0) - np.float32(1.5) * dphi - np.float32(1e-4) * np.arange(N)
    w.standin(st, 0.0, 0.0)
    w.env_step(st, prev_action=np.zeros((N, w.A), np.float32))
    assert not st.truncated.any() and not st.terminated.any()
    Plast, Qlast, _, _ = w.ref_state(0, np.float32(1.0))
    leaves = _leaves(d)
    D0 = 15 * w.B + 1
    for e in range(N):
        HT, org = _heading(st.quat[0, :, e].astype(np.float64), st.pos[0, :, e].astype(np.float64))
        ph1 = np.float32(st.phase[e] + dphi)
        assert ph1 >= 1.0
        idx = D0
        for j in range(d["config"]["obs_future"]):
            for b in [0] + leaves:
                np.testing.assert_allclose(st.obs[idx:idx + 9, e],
                                           _frame9(HT, org, Plast[b], Qlast[b]), atol=2e-6)
                idx += 9
