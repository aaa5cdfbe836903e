"""Pins of the tracking reward and the termination rule."""
import math

import numpy as np
import pytest

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


def test_without_ee_weight_is_the_three_term_reward():
    # Sec. 4.1 / Fig. 5: the tracking reward is a weighted sum of three
    # exponentiated errors -- the squared body-position differences summed over
    # bodies and axes, the same for the body velocities, and the squared
    # distance between the mass-weighted centres of the simulated and reference
    # bodies -- with weights 0.60 / 0.25 / 0.15 and scales 4 / 0.25 / 8.  With
    # the end-effector weight at zero the oracle's reward is that sum, written
    # out here per body from the definition.
    d = synth.make_world(2, n_envs=1, w_ee=0.0)
    cfg = d["config"]
    assert (cfg["c_pose"], cfg["w_pos"], cfg["c_vel"], cfg["w_vel"], cfg["c_com"], cfg["w_com"]) == \
        (np.float32(0.60), 4.0, np.float32(0.25), 0.25, np.float32(0.15), 8.0)
    w = oracle.World(d)
    P, V = _ref(w)
    m, M = _masses(d)
    for _ in range(10):
        Ps = P + RNG.normal(size=P.shape) * 0.05
        Vs = V + RNG.normal(size=V.shape) * 0.5
        pose = vel = 0.0
        csim, cref = [0.0, 0.0, 0.0], [0.0, 0.0, 0.0]
        for b in range(w.B):
            for c in range(3):
                pose += (float(Ps[b, c]) - float(P[b, c])) ** 2
                vel += (float(Vs[b, c]) - float(V[b, c])) ** 2
                csim[c] += float(m[b]) * float(Ps[b, c]) / M
                cref[c] += float(m[b]) * float(P[b, c]) / M
        com = sum((csim[c] - cref[c]) ** 2 for c in range(3))
        # the weights and scales are float32 fields of the step configuration
        f = lambda k: float(np.float32(cfg[k]))
        expect = (f("c_pose") * math.exp(-f("w_pos") * pose) + f("c_vel") * math.exp(-f("w_vel") * vel)
                  + f("c_com") * math.exp(-f("w_com") * com))
        assert w.reward(Ps, Vs, P, V)["r"] == pytest.approx(expect, rel=1e-12)


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
