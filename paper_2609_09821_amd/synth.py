"""Seeded synthetic inputs: skeletons, reference clips, policy weights, configs.

This module only makes input data.  It holds none of the step's arithmetic
(no sampling, kinematics, reward, observation or policy math) and imports
neither the HIP binding nor the oracle, so both consume the same arrays.

The paper trains on its own mocap clips and a MuJoCo humanoid model, neither
of which is available; these generators stand in for them with the shapes of
the benchmark workloads:

* S15 -- 15-body humanoid: root (free joint), 8 spherical, 4 revolute (about
  the local +y axis), 2 fixed joints, action width 28, observation 226.
* S24 -- 24-body SMPL-like tree, all spherical: action 69, observation 361.
* Clips at 30 fps: every joint DoF follows a sum of three sinusoids with
  amplitudes drawn so |angle| <= 0.8 rad; the root moves forward at 1 m/s at
  0.9 m height with a small (<= 0.2 rad per axis) sinusoidal orientation
  wobble so that the heading varies.
* Policy weights: U(-1/sqrt(fan_in), 1/sqrt(fan_in)), bf16 configurations
  store them already rounded to bf16.
"""
from __future__ import annotations

import numpy as np

JT_FREE, JT_SPH, JT_REV, JT_FIXED = 0, 1, 2, 3

# (name, parent, joint type, canonical offset direction in the parent frame)
_S15 = [
    ("root", -1, JT_FREE, (0, 0, 0)),
    ("chest", 0, JT_SPH, (0, 0, 1)),
    ("neck", 1, JT_SPH, (0, 0, 1)),
    ("r_hip", 0, JT_SPH, (0, -1, 0)),
    ("r_knee", 3, JT_REV, (0, 0, -1)),
    ("r_ankle", 4, JT_SPH, (0, 0, -1)),
    ("r_shoulder", 1, JT_SPH, (0, -1, 0)),
    ("r_elbow", 6, JT_REV, (0, -1, 0)),
    ("r_wrist", 7, JT_FIXED, (0, -1, 0)),
    ("l_hip", 0, JT_SPH, (0, 1, 0)),
    ("l_knee", 9, JT_REV, (0, 0, -1)),
    ("l_ankle", 10, JT_SPH, (0, 0, -1)),
    ("l_shoulder", 1, JT_SPH, (0, 1, 0)),
    ("l_elbow", 12, JT_REV, (0, 1, 0)),
    ("l_wrist", 13, JT_FIXED, (0, 1, 0)),
]

_S24 = [
    ("pelvis", -1, JT_FREE, (0, 0, 0)),
    ("l_hip", 0, JT_SPH, (0, 1, 0)),
    ("r_hip", 0, JT_SPH, (0, -1, 0)),
    ("spine1", 0, JT_SPH, (0, 0, 1)),
    ("l_knee", 1, JT_SPH, (0, 0, -1)),
    ("r_knee", 2, JT_SPH, (0, 0, -1)),
    ("spine2", 3, JT_SPH, (0, 0, 1)),
    ("l_ankle", 4, JT_SPH, (0, 0, -1)),
    ("r_ankle", 5, JT_SPH, (0, 0, -1)),
    ("spine3", 6, JT_SPH, (0, 0, 1)),
    ("l_foot", 7, JT_SPH, (1, 0, 0)),
    ("r_foot", 8, JT_SPH, (1, 0, 0)),
    ("neck", 9, JT_SPH, (0, 0, 1)),
    ("l_collar", 9, JT_SPH, (0, 1, 0)),
    ("r_collar", 9, JT_SPH, (0, -1, 0)),
    ("head", 12, JT_SPH, (0, 0, 1)),
    ("l_shoulder", 13, JT_SPH, (0, 1, 0)),
    ("r_shoulder", 14, JT_SPH, (0, -1, 0)),
    ("l_elbow", 16, JT_SPH, (0, 1, 0)),
    ("r_elbow", 17, JT_SPH, (0, -1, 0)),
    ("l_wrist", 18, JT_SPH, (0, 1, 0)),
    ("r_wrist", 19, JT_SPH, (0, -1, 0)),
    ("l_hand", 20, JT_SPH, (0, 1, 0)),
    ("r_hand", 21, JT_SPH, (0, -1, 0)),
]


def _skeleton(table, rng):
    B = len(table)
    parent = np.array([t[1] for t in table], np.int32)
    jtype = np.array([t[2] for t in table], np.int32)
    axis = np.zeros((B, 3), np.float32)
    axis[jtype == JT_REV] = (0.0, 1.0, 0.0)
    lengths = rng.uniform(0.1, 0.45, size=B)
    offset = np.array([np.asarray(t[3], np.float64) * lengths[i] for i, t in enumerate(table)])
    offset[0] = 0.0
    mass = rng.uniform(1.0, 10.0, size=B)
    return dict(
        name="S%d" % B,
        n_bodies=B,
        names=[t[0] for t in table],
        parent=parent,
        jtype=jtype,
        axis=axis,
        offset=offset.astype(np.float32),
        mass=mass.astype(np.float32),
    )


def skeleton_s15(rng):
    return _skeleton(_S15, rng)


def skeleton_s24(rng):
    return _skeleton(_S24, rng)


def _quat_from_rotvec(r):
    """Unit quaternion (w,x,y,z) of rotation vectors r[..., 3] (input data)."""
    r = np.asarray(r, np.float64)
    th = np.linalg.norm(r, axis=-1, keepdims=True)
    half = 0.5 * th
    with np.errstate(invalid="ignore", divide="ignore"):
        k = np.where(th > 0, np.sin(half) / np.where(th > 0, th, 1.0), 0.5)
    q = np.concatenate([np.cos(half), r * k], axis=-1)
    return q / np.linalg.norm(q, axis=-1, keepdims=True)


def _sinusoid_sum(rng, n_dof, times, amp_total):
    """n_dof signals sum_{k<3} a_k sin(2 pi f_k t + psi_k), |signal| <= amp_total."""
    a = rng.uniform(-amp_total / 3.0, amp_total / 3.0, size=(n_dof, 3))
    f = rng.uniform(0.2, 1.5, size=(n_dof, 3))
    psi = rng.uniform(0.0, 2.0 * np.pi, size=(n_dof, 3))
    t = times[:, None, None]
    return np.sum(a * np.sin(2.0 * np.pi * f * t + psi), axis=-1)  # [F][n_dof]


def make_clip(rng, skel, n_frames, fps=30.0, joint_amp=0.8, root_amp=0.2, speed=1.0,
              height=0.9):
    B = skel["n_bodies"]
    jt = skel["jtype"]
    times = np.arange(n_frames, dtype=np.float64) / fps
    root_pos = np.stack([speed * times, np.zeros_like(times), np.full_like(times, height)], -1)
    root_rv = _sinusoid_sum(rng, 3, times, root_amp)
    root_quat = _quat_from_rotvec(root_rv)
    local = np.zeros((n_frames, B - 1, 4), np.float64)
    local[..., 0] = 1.0
    for b in range(1, B):
        if jt[b] == JT_SPH:
            rv = _sinusoid_sum(rng, 3, times, joint_amp)
            local[:, b - 1] = _quat_from_rotvec(rv)
        elif jt[b] == JT_REV:
            ang = _sinusoid_sum(rng, 1, times, joint_amp)
            local[:, b - 1] = _quat_from_rotvec(ang * skel["axis"][b].astype(np.float64))
    return dict(
        n_frames=int(n_frames),
        fps=float(fps),
        root_pos=root_pos.astype(np.float32),
        root_quat=root_quat.astype(np.float32),
        local_quat=local.astype(np.float32),
    )


def bf16_round(x):
    """Round float32 values to the nearest bf16 (ties to even), kept in float32."""
    x = np.ascontiguousarray(x, np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    out = r.astype(np.uint32).view(np.float32)
    return np.where(np.isfinite(x), out, x).astype(np.float32)


def make_policy(rng, dims, bf16, sigma=0.05):
    W, b = [], []
    for i in range(len(dims) - 1):
        fan_in, fan_out = dims[i], dims[i + 1]
        lim = 1.0 / np.sqrt(fan_in)
        w = rng.uniform(-lim, lim, size=(fan_out, fan_in)).astype(np.float32)
        bb = rng.uniform(-lim, lim, size=fan_out).astype(np.float32)
        if bf16:
            w = bf16_round(w)
        W.append(np.ascontiguousarray(w))
        b.append(np.ascontiguousarray(bb))
    log_std = np.full(dims[-1], np.log(sigma), np.float32)
    return dict(dims=list(dims), bf16=bool(bf16), W=W, b=b, log_std=log_std)


# The five benchmark workloads.  Seeds: master = workload id.
R_MIN_6 = 0.587   # the oracle's 20th-percentile reward of this workload (3 s.f.)

CONFIGS = {
    1: dict(name="S15 64 envs single step, fp32 MLP 226-1024-512-28", n_envs=64, skeleton="S15",
            frames=[30], mlp=[226, 1024, 512, 28], bf16=False, steps=1, sigma_joint=0.05),
    2: dict(name="S15 4096 envs 32-step rollout, 120-frame clip, fp32 MLP 226-1024-512-28",
            n_envs=4096, skeleton="S15", frames=[120], mlp=[226, 1024, 512, 28], bf16=False,
            steps=32, sigma_joint=0.05),
    3: dict(name="S15 16384 envs 32-step rollout, 3 clips (60/150/90), bf16 MLP 226-1024-512-28",
            n_envs=16384, skeleton="S15", frames=[60, 150, 90], mlp=[226, 1024, 512, 28],
            bf16=True, steps=32, sigma_joint=0.05),
    4: dict(name="S24 65536 envs 32-step rollout, 300-frame clip, bf16 MLP 361-1024-1024-512-69",
            n_envs=65536, skeleton="S24", frames=[300], mlp=[361, 1024, 1024, 512, 69],
            bf16=True, steps=32, sigma_joint=0.05),
    5: dict(name="S15 262144 envs 16-step rollout, 16 clips of 60-300 frames, sigma_joint 0.3, "
                 "bf16 MLP 226-1024-512-28",
            n_envs=262144, skeleton="S15", frames="16x60-300", mlp=[226, 1024, 512, 28],
            bf16=True, steps=16, sigma_joint=0.3),
    # the training step's terms: multiplicative 5-term reward (joint rotation 10, COM 10 and
    # end-effector orientation 2 as in the configuration table; joint velocity 0.1 and
    # end-effector position 40 read from DeepMimic's scales), termination height 0.8 and
    # 4 grace steps (table baseline), 2 future reference frames and the previous action in
    # the observation (D = 361 + 2*6*9 + 69 = 538)
    6: dict(name="S24 16384 envs 32-step rollout, 300-frame clip, multiplicative reward, "
                 "observation with 2 future frames + previous action, bf16 MLP 538-1024-1024-512-69",
            n_envs=16384, skeleton="S24", frames=[300], mlp=[538, 1024, 1024, 512, 69],
            bf16=True, steps=32, sigma_joint=0.01, sigma_vel=0.1,
            config=dict(reward_form=1, h_term=0.8, grace=4, r_min=R_MIN_6,
                        obs_future=2, obs_prev_action=1)),
}

SEED_BASE = 0x0A11_2609_0982_1000


def step_config(master, **over):
    cfg = dict(
        dt=1.0 / 30.0,
        h_term=0.3,
        r_min=0.15,
        grace=0,
        c_pose=0.60, w_pos=4.0, w_ee=40.0,
        c_vel=0.25, w_vel=0.25,
        c_com=0.15, w_com=8.0,
        seed=SEED_BASE + int(master),
        # training terms: reward_form 1 = multiplicative reward with weights
        # m_jrot, m_jvel, m_com, m_eepos, m_eerot; obs_future reference frames
        # and the previous action in the observation
        reward_form=0,
        m_jrot=10.0, m_jvel=0.1, m_com=10.0, m_eepos=40.0, m_eerot=2.0,
        obs_future=0, obs_prev_action=0,
    )
    cfg.update(CONFIGS.get(int(master), {}).get("config", {}))
    cfg.update(over)
    return cfg


def obs_dim(n_bodies, n_ee, n_actions, cfg):
    """Observation width: 15 rows per body, the phase, 9 per future reference
    frame of the root and each end effector, the previous action."""
    return (15 * n_bodies + 1 + int(cfg["obs_future"]) * (1 + n_ee) * 9
            + (n_actions if cfg["obs_prev_action"] else 0))


def make_world(cfg_id, n_envs=None, **cfg_over):
    """Everything both implementations need for workload `cfg_id`."""
    spec = dict(CONFIGS[cfg_id])
    ss = np.random.SeedSequence(cfg_id).spawn(4)
    r_skel, r_clip, r_pol, r_crit = (np.random.default_rng(s) for s in ss)
    skel = skeleton_s15(r_skel) if spec["skeleton"] == "S15" else skeleton_s24(r_skel)
    if spec["frames"] == "16x60-300":
        frames = [int(f) for f in r_clip.integers(60, 301, size=16)]
    else:
        frames = list(spec["frames"])
    clips = [make_clip(r_clip, skel, F) for F in frames]
    pol = make_policy(r_pol, spec["mlp"], spec["bf16"])
    # value head: the policy's hidden widths, one output
    critic = make_policy(r_crit, list(spec["mlp"][:-1]) + [1], spec["bf16"])
    cfg = step_config(cfg_id, **cfg_over)
    return dict(
        id=cfg_id,
        spec=spec,
        n_envs=int(n_envs if n_envs is not None else spec["n_envs"]),
        skeleton=skel,
        clips=clips,
        policy=pol,
        critic=critic,
        config=cfg,
        sigma_joint=float(spec["sigma_joint"]),
        sigma_vel=float(spec.get("sigma_vel", 0.5)),
    )


# PPO rollout-end parameters: discount and GAE lambda (baseline column of the
# backflip configuration table)
GAMMA, LAMBDA = 0.99, 0.95


def rollout_inputs(seed, T, N, p_term=0.04, p_trunc=0.02):
    """Seeded stand-ins for a rollout's stored rewards, flags and values:
    reward U(0, 1), terminated / truncated Bernoulli(p_term / p_trunc) (both
    may be set), values N(0, 2^2) for the T + 1 observations, running-episode
    return U(0, 5) and length 0..49 from earlier rollouts."""
    rng = np.random.default_rng(np.random.SeedSequence([2609, seed]))
    reward = rng.uniform(0.0, 1.0, size=(T, N)).astype(np.float32)
    term = (rng.random((T, N)) < p_term).astype(np.uint8)
    trunc = (rng.random((T, N)) < p_trunc).astype(np.uint8)
    value = (2.0 * rng.standard_normal((T + 1, N))).astype(np.float32)
    ep_return = rng.uniform(0.0, 5.0, size=N).astype(np.float32)
    ep_length = rng.integers(0, 50, size=N).astype(np.int32)
    return dict(reward=reward, term=term, trunc=trunc, value=value, ep_return=ep_return,
                ep_length=ep_length)
