"""Shared helpers of the GPU parity tests: moving oracle.State <-> device
buffers, and the comparison rules (tolerances written out here).

Tolerances:
* discrete env state (clip, phase, t, n), flags, reference frame index:
  bit-exact (flags: except where the oracle's reward lies within the reward
  tolerance of r_min, where both decisions are correct; such envs are
  excluded from later steps);
* reward: |g - o| <= 1e-5 |o| + 1e-6;
* observations and reference-state sim writes: |g - o| <= 1e-5 max(|o|, 1),
  quaternions compared up to sign;
* policy: per env ||g - o||_2 <= 2e-2 ||o||_2 for bf16 weights/activations,
  <= 1e-4 ||o||_2 for fp32; logp |g - o| <= 1e-5 |o| + 1e-4.
"""
import numpy as np
import torch

import oracle
from paper_2609_09821_amd import binding

REW_RTOL, REW_ATOL = 1e-5, 1e-6
OBS_TOL = 1e-5


def upload_state(st: "oracle.State", bufs: binding.EnvBuffers, sim=True, env=True):
    if env:
        bufs.env_clip[:st.N].copy_(torch.from_numpy(st.clip))
        bufs.env_phase[:st.N].copy_(torch.from_numpy(st.phase))
        bufs.env_t[:st.N].copy_(torch.from_numpy(st.t))
        bufs.env_n[:st.N].copy_(torch.from_numpy(st.n.view(np.int32)))
    if sim:
        for name, arr in (("body_pos", st.pos), ("body_quat", st.quat),
                          ("body_linvel", st.linvel), ("body_angvel", st.angvel)):
            getattr(bufs, name)[:, :, :st.N].copy_(torch.from_numpy(arr))


def download(bufs: binding.EnvBuffers, N):
    torch.cuda.synchronize()
    g = oracle.State(bufs.B, N)
    g.clip = bufs.env_clip[:N].cpu().numpy()
    g.phase = bufs.env_phase[:N].cpu().numpy()
    g.t = bufs.env_t[:N].cpu().numpy()
    g.n = bufs.env_n[:N].cpu().numpy().view(np.uint32)
    g.pos = np.ascontiguousarray(bufs.body_pos[:, :, :N].cpu().numpy())
    g.quat = np.ascontiguousarray(bufs.body_quat[:, :, :N].cpu().numpy())
    g.linvel = np.ascontiguousarray(bufs.body_linvel[:, :, :N].cpu().numpy())
    g.angvel = np.ascontiguousarray(bufs.body_angvel[:, :, :N].cpu().numpy())
    g.reward = bufs.reward[:N].cpu().numpy()
    g.terminated = bufs.terminated[:N].cpu().numpy()
    g.truncated = bufs.truncated[:N].cpu().numpy()
    g.obs = np.ascontiguousarray(bufs.obs[:, :N].cpu().numpy())
    g.ref_frame = bufs.ref_frame[:N].cpu().numpy()
    return g


def assert_close(g, o, tol=OBS_TOL, what="", idx=None):
    g = np.asarray(g, np.float64)
    o = np.asarray(o, np.float64)
    err = np.abs(g - o) / np.maximum(np.abs(o), 1.0)
    bad = ~(err <= tol)
    if bad.any():
        where = np.argwhere(bad)[:5]
        raise AssertionError("%s: %d values out of tolerance %.1e; worst %.3e at %s; e.g. g=%s o=%s"
                             % (what, int(bad.sum()), tol, float(np.nanmax(err)),
                                where.tolist(), g[tuple(where[0])], o[tuple(where[0])]))


def assert_quat_close(g, o, tol=OBS_TOL, what=""):
    # [B][4][N]: align signs per (body, env)
    s = np.sign((g.astype(np.float64) * o).sum(axis=1, keepdims=True))
    s[s == 0] = 1
    assert_close(g * s, o, tol, what)


def reward_ok(g, o):
    g = np.asarray(g, np.float64)
    o = np.asarray(o, np.float64)
    return np.abs(g - o) <= REW_RTOL * np.abs(o) + REW_ATOL


def compare_step(g, o, r_min, h_term, grace, t_next, z_root, live):
    """Compare one step's outputs on the `live` envs; returns the new live mask."""
    assert np.array_equal(g.ref_frame[live], o.ref_frame[live]), "reference frame index differs"
    ok = reward_ok(g.reward, o.reward)
    bad = live & ~ok
    assert not bad.any(), "reward out of tolerance at envs %s: g=%s o=%s" % (
        np.flatnonzero(bad)[:5], g.reward[bad][:5], o.reward[bad][:5])
    # the GPU's flags follow its own reward exactly
    exp_term = (t_next > grace) & ((z_root < np.float32(h_term)) | ~(g.reward >= np.float32(r_min)))
    assert np.array_equal(g.terminated[live].astype(bool), exp_term[live]), "GPU flag rule"
    assert np.array_equal(g.truncated[live], o.truncated[live]), "truncation differs"
    tie = (g.terminated != o.terminated)
    band = np.abs(o.reward.astype(np.float64) - r_min) <= REW_RTOL * abs(r_min) + REW_ATOL
    assert not (live & tie & ~band).any(), "termination differs away from the threshold"
    live = live & ~tie
    for name in ("clip", "phase", "t", "n"):
        assert np.array_equal(getattr(g, name)[live], getattr(o, name)[live]), name + " differs"
    return live


def compare_sim_obs(g, o, live, what=""):
    assert_close(g.pos[:, :, live], o.pos[:, :, live], what=what + " body_pos")
    assert_quat_close(g.quat[:, :, live], o.quat[:, :, live], what=what + " body_quat")
    assert_close(g.linvel[:, :, live], o.linvel[:, :, live], what=what + " body_linvel")
    assert_close(g.angvel[:, :, live], o.angvel[:, :, live], what=what + " body_angvel")
    assert_close(g.obs[:, live], o.obs[:, live], what=what + " obs")
