"""Pins of the composed step: reset draws, RSI, masked reset, the stand-in."""
import numpy as np
import pytest
from scipy import stats

import oracle
from paper_2609_09821_amd import synth


def _philox_key(seed):
    return [seed & 0xFFFFFFFF, seed >> 32]


def test_reset_draw_uses_philox_words():
    d = synth.make_world(5, n_envs=1)
    w = oracle.World(d)
    C = len(d["clips"])
    for e in range(200):
        for tag in (1, 4):
            x = oracle.philox([e, 9, 0, tag], _philox_key(w.seed))
            k, phi = w.reset_draw(e, 9, tag)
            assert k == (int(x[0]) * C) >> 32
            assert phi == np.float32((int(x[1]) >> 8) / 2.0 ** 24)
            assert 0 <= k < C and np.float32(0) <= phi < np.float32(1)


def test_reset_draw_uniformity():
    d = synth.make_world(5, n_envs=1)
    w = oracle.World(d)
    C = len(d["clips"])
    ks, phis = [], []
    for e in range(20000):
        k, p = w.reset_draw(e, 3, 1)
        ks.append(k)
        phis.append(float(p))
    counts = np.bincount(ks, minlength=C)
    assert stats.chisquare(counts).pvalue > 1e-3
    assert stats.kstest(phis, "uniform").pvalue > 1e-3


@pytest.mark.parametrize("cfg", [1, 4])
def test_reset_envs_writes_reference_state(cfg):
    d = synth.make_world(cfg, n_envs=50)
    w = oracle.World(d)
    st = oracle.State(w.B, 50)
    st.n[:] = np.arange(50, dtype=np.uint32) * 7
    w.reset_envs(st)
    for e in range(50):
        k, phi = w.reset_draw(e, int(st.n[e]), 4)
        assert st.clip[e] == k and st.phase[e] == phi and st.t[e] == 0
        P, Q, V, W = w.ref_state(k, phi)
        np.testing.assert_array_equal(st.pos[:, :, e], P.astype(np.float32))
        np.testing.assert_array_equal(st.quat[:, :, e], Q.astype(np.float32))
        np.testing.assert_array_equal(st.linvel[:, :, e], V.astype(np.float32))
        np.testing.assert_array_equal(st.angvel[:, :, e], W.astype(np.float32))
        assert st.obs[-1, e] == phi


def test_reset_envs_mask_leaves_others_untouched():
    d = synth.make_world(2, n_envs=64)
    w = oracle.World(d)
    st = oracle.State(w.B, 64)
    w.reset_envs(st)
    before = st.copy()
    mask = np.zeros(64, np.uint8)
    mask[::3] = 1
    st.n[:] += 5
    w.reset_envs(st, mask)
    for e in range(64):
        same = (np.array_equal(st.pos[:, :, e], before.pos[:, :, e])
                and st.phase[e] == before.phase[e])
        assert same == (not mask[e])


@pytest.mark.parametrize("cfg", [2, 4])
def test_noise_free_standin_gives_reward_one(cfg):
    # sim = reference (rounded to fp32) -> every error is below 2^-25, exp rounds to 1
    d = synth.make_world(cfg, n_envs=40)
    w = oracle.World(d)
    st = oracle.State(w.B, 40)
    w.reset_envs(st)
    w.standin(st, 0.0, 0.0)
    w.env_step(st)
    np.testing.assert_array_equal(st.reward, np.float32(1.0))
    assert not st.terminated.any()


def test_standin_noise_statistics():
    d = synth.make_world(2, n_envs=3000)
    w = oracle.World(d)
    st = oracle.State(w.B, 3000)
    w.reset_envs(st)
    ref = st.copy()
    w.standin(ref, 0.0, 0.0)
    w.standin(st, 0.05, 0.5)
    dv = (st.linvel - ref.linvel).reshape(-1) / 0.5
    dw = (st.angvel - ref.angvel).reshape(-1) / 0.5
    for z in (dv, dw):
        assert abs(z.mean()) < 0.01 and abs(z.std() - 1) < 0.01
    # the root position is not perturbed, the root orientation is
    np.testing.assert_array_equal(st.pos[0], ref.pos[0])
    ang = 2 * np.arccos(np.clip(np.abs((st.quat[0] * ref.quat[0]).sum(0)), 0, 1))
    # angle of a 3D isotropic normal rotation vector, sigma 0.05: mean 0.05*sqrt(8/pi)
    assert abs(ang.mean() - 0.05 * np.sqrt(8 / np.pi)) < 0.003


def test_step_advances_and_resets():
    d = synth.make_world(3, n_envs=300)
    w = oracle.World(d)
    st = oracle.State(w.B, 300)
    w.reset_envs(st)
    st.phase[:5] = np.float32(0.9999)  # forces truncation
    prev = st.copy()
    w.standin(st, d["sigma_joint"], d["sigma_vel"])
    sim_in = st.copy()
    w.env_step(st)
    for e in range(300):
        k = prev.clip[e]
        phi1 = np.float32(prev.phase[e] + w.dphi(k))
        assert st.truncated[e] == (phi1 >= 1)
        assert st.n[e] == prev.n[e] + 1
        done = st.truncated[e] or st.terminated[e]
        if done:
            kk, pp = w.reset_draw(e, int(prev.n[e]) + 1, 1)
            assert st.clip[e] == kk and st.phase[e] == pp and st.t[e] == 0
        else:
            assert st.clip[e] == k and st.phase[e] == phi1 and st.t[e] == prev.t[e] + 1
            np.testing.assert_array_equal(st.pos[:, :, e], sim_in.pos[:, :, e])
        assert st.obs[-1, e] == st.phase[e]
    assert st.truncated[:5].all()


def test_step_root_below_height_terminates():
    d = synth.make_world(2, n_envs=20, h_term=0.3)
    w = oracle.World(d)
    st = oracle.State(w.B, 20)
    w.reset_envs(st)
    w.standin(st, 0.0, 0.0)
    st.pos[0, 2, :10] = np.float32(0.29)
    st.pos[0, 2, 10:] = np.float32(0.3)
    w.env_step(st)
    assert st.terminated[:10].all() and not st.terminated[10:].any()


def test_standin_local_rotation_noise():
    # recover each joint's local noise rotation from the world orientations:
    # delta_b = (Q_p^-1 Q_b)_ref^-1 (Q_p^-1 Q_b)_noisy; spherical joints: every
    # rotation-vector component ~ N(0, sigma^2); revolute: only about the axis;
    # fixed: none
    from scipy.spatial.transform import Rotation
    N, sig = 4000, 0.05
    d = synth.make_world(2, n_envs=N)
    w = oracle.World(d)
    st = oracle.State(w.B, N)
    w.reset_envs(st)
    ref = st.copy()
    w.standin(ref, 0.0, 0.0)
    w.standin(st, sig, 0.5)
    sk = d["skeleton"]
    R = lambda q: Rotation.from_quat(np.stack([q[1], q[2], q[3], q[0]], -1))
    for b in range(1, w.B):
        p = sk["parent"][b]
        loc_n = R(st.quat[p]).inv() * R(st.quat[b])
        loc_r = R(ref.quat[p]).inv() * R(ref.quat[b])
        rv = (loc_r.inv() * loc_n).as_rotvec() / sig
        if sk["jtype"][b] == synth.JT_SPH:
            assert np.all(np.abs(rv.mean(0)) < 0.08) and np.all(np.abs(rv.std(0) - 1) < 0.06)
        elif sk["jtype"][b] == synth.JT_REV:
            ax = sk["axis"][b].astype(np.float64)
            along = rv @ ax
            assert abs(along.std() - 1) < 0.06
            assert np.abs(rv - np.outer(along, ax)).max() < 1e-3
        else:
            assert np.abs(rv).max() < 1e-3
    root = (R(ref.quat[0]).inv() * R(st.quat[0])).as_rotvec() / sig
    assert np.all(np.abs(root.std(0) - 1) < 0.06)


def test_step_non_finite_state_terminates_and_resets():
    # a NaN anywhere in the read sim state makes the reward NaN, which fails r >= r_min
    d = synth.make_world(2, n_envs=30)
    w = oracle.World(d)
    st = oracle.State(w.B, 30)
    w.reset_envs(st)
    w.standin(st, d["sigma_joint"], d["sigma_vel"])
    st.pos[4, 0, 0:10] = np.nan
    st.linvel[7, 2, 10:20] = np.nan
    prev_n = st.n.copy()
    w.env_step(st)
    assert np.all(np.isnan(st.reward[:20])) and np.all(np.isfinite(st.reward[20:]))
    assert st.terminated[:20].all()
    for e in range(20):
        k, p = w.reset_draw(e, int(prev_n[e]) + 1, 1)
        assert st.clip[e] == k and st.phase[e] == p and st.t[e] == 0
    assert np.all(np.isfinite(st.obs[:, :20])) and np.all(np.isfinite(st.pos[:, :, :20]))
