"""Pins of the tracking reward and the termination rule."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_09821_amd import synth

RNG = np.random.default_rng(5)


@pytest.fixture(scope="module", params=[2, 4])
def world(request):
    d = synth.make_world(request.param, n_envs=1)
    return d, oracle.World(d)


def _ref(w, phi=0.37):
    P, Q, V, W = w.ref_state(0, np.float32(phi))
    return P, V


def test_zero_error_reward_is_exactly_one(world):
    d, w = world
    P, V = _ref(w)
    r = w.reward(P, V, P, V)
    assert r["e_pos"] == r["e_vel"] == r["e_ee"] == r["e_com"] == 0.0
    assert np.float32(r["r"]) == np.float32(1.0)


def _masses(d):
    m = d["skeleton"]["mass"].astype(np.float64)
    return m, m.sum()


def _leaves(d):
    par = d["skeleton"]["parent"]
    return [b for b in range(len(par)) if b not in set(par[1:])]


def test_single_body_displacement_closed_form(world):
    d, w = world
    P, V = _ref(w)
    m, M = _masses(d)
    leaves = _leaves(d)
    cfg = d["config"]
    for b in range(w.B):
        dp = RNG.normal(size=3) * 0.1
        Ps = P.copy()
        Ps[b] += dp
        r = w.reward(Ps, V, P, V)
        x = float(dp @ dp)
        e_ee = x if b in leaves else 0.0
        e_com = (m[b] / M) ** 2 * x
        expect = (np.float32(cfg["c_pose"]) * np.exp(-(4.0 * x + 40.0 * e_ee))
                  + np.float32(cfg["c_vel"]) + np.float32(cfg["c_com"]) * np.exp(-8.0 * e_com))
        assert r["e_pos"] == pytest.approx(x, rel=1e-12)
        assert r["e_ee"] == pytest.approx(e_ee, rel=1e-12, abs=1e-300)
        assert r["e_com"] == pytest.approx(e_com, rel=1e-9)
        assert r["r"] == pytest.approx(expect, rel=1e-12)


def test_velocity_only_closed_form(world):
    d, w = world
    P, V = _ref(w)
    Vs = V + RNG.normal(size=V.shape) * 0.3
    r = w.reward(P, Vs, P, V)
    x = float(((Vs - V) ** 2).sum())
    expect = np.float32(0.60) + np.float32(0.25) * np.exp(-0.25 * x) + np.float32(0.15)
    assert r["e_vel"] == pytest.approx(x, rel=1e-12)
    assert r["r"] == pytest.approx(expect, rel=1e-12)


def test_rigid_translation_moves_only_position_terms(world):
    # a rigid shift of every body by d: e_pos = B|d|^2, e_ee = n_leaves|d|^2, e_com = |d|^2
    d, w = world
    P, V = _ref(w)
    sh = np.array([0.03, -0.02, 0.01])
    r = w.reward(P + sh, V, P, V)
    x = float(sh @ sh)
    assert r["e_pos"] == pytest.approx(w.B * x, rel=1e-9)
    assert r["e_ee"] == pytest.approx(len(_leaves(d)) * x, rel=1e-9)
    assert r["e_com"] == pytest.approx(x, rel=1e-9)


def test_without_ee_weight_equals_fig5_reward():
    # The paper's printed tensor code (Fig. 5a), transcribed; with the EE weight at
    # zero the oracle's reward is that three-term form.
    d = synth.make_world(2, n_envs=1, w_ee=0.0)
    w = oracle.World(d)
    P, V = _ref(w)
    m, M = _masses(d)
    for _ in range(10):
        Ps = P + RNG.normal(size=P.shape) * 0.05
        Vs = V + RNG.normal(size=V.shape) * 0.5
        body_pos, ref_body_pos = torch.tensor(Ps)[None], torch.tensor(P)[None]
        body_vel, ref_body_vel = torch.tensor(Vs)[None], torch.tensor(V)[None]
        mt = torch.tensor(m)[:, None]
        com_pos = (mt * body_pos[0]).sum(0, keepdim=True) / M
        ref_com_pos = (mt * ref_body_pos[0]).sum(0, keepdim=True) / M
        pose_err = (body_pos - ref_body_pos).square().sum(dim=(-1, -2))
        vel_err = (body_vel - ref_body_vel).square().sum(dim=(-1, -2))
        com_err = (com_pos - ref_com_pos).square().sum(dim=-1)
        reward = (float(np.float32(0.60)) * torch.exp(-4.0 * pose_err)
                  + 0.25 * torch.exp(-0.25 * vel_err)
                  + float(np.float32(0.15)) * torch.exp(-8.0 * com_err))
        assert w.reward(Ps, Vs, P, V)["r"] == pytest.approx(float(reward[0]), rel=1e-12)


def test_termination_truth_table():
    d = synth.make_world(2, n_envs=1, h_term=0.55, r_min=0.15, grace=0)
    w = oracle.World(d)
    h, rm = np.float32(0.55), np.float32(0.15)
    up = np.nextafter(h, np.float32(1))
    dn = np.nextafter(h, np.float32(0))
    assert not w.terminated(1, h, 0.9)          # equality is not below (strict <)
    assert w.terminated(1, dn, 0.9)
    assert not w.terminated(1, up, 0.9)
    assert not w.terminated(1, 0.9, rm)          # reward equal to the threshold survives
    assert w.terminated(1, 0.9, np.nextafter(rm, np.float32(0)))
    assert w.terminated(1, 0.9, np.float32("nan"))  # a non-finite reward terminates
    assert w.terminated(1, np.float32(0.1), np.float32(0.1))


def test_termination_grace_steps():
    d = synth.make_world(2, n_envs=1, grace=4)
    w = oracle.World(d)
    for t in range(0, 5):
        assert not w.terminated(t, 0.0, 0.0)
    assert w.terminated(5, 0.0, 0.0)
