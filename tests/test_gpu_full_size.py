"""Parity at the full workload sizes, in the launch configuration the bench
times (ld = n_envs, 256-env blocks of the env kernel, the large-batch GEMM
tiles of the policy).

Every env is compared with the oracle: the env step (reset and teacher-forced
steps), the policy (mean, action and logp of all 65536 / 262144 / 16384 envs,
so every GEMM tile and the env tail) and the critic.  The policy is also
checked through properties that hold at any size: finite outputs, logp equal
to the value implied by the env's own (action - mean) / sigma, and
standard-normal noise statistics over the whole batch.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_09821_amd import binding, synth
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu

FULL = {4: 2, 5: 2, 6: 6}    # workload -> teacher-forced steps (6: past its grace period)


@pytest.fixture(scope="module", params=[4, 5, 6])
def world(request):
    cfg = request.param
    d = synth.make_world(cfg)
    N = d["n_envs"]
    w = oracle.World(d)
    ctx = binding.Context(d, max_envs=N)
    bufs = ctx.buffers(N)
    print("full-size world cfg %d: %d envs" % (cfg, N), flush=True)
    yield cfg, d, w, ctx, bufs
    ctx.close()


def test_full_size_env_step(world):
    cfg, d, w, ctx, bufs = world
    N = d["n_envs"]
    c = d["config"]
    st = w.state(N)
    w.reset_envs(st)
    ctx.reset_envs(bufs)
    g = H.download(bufs, N)
    for name in ("clip", "phase", "t", "n"):
        assert np.array_equal(getattr(g, name), getattr(st, name)), name
    H.compare_sim_obs(g, st, np.ones(N, bool), "full-size reset")
    live = np.ones(N, bool)
    n_done = 0
    rng = np.random.default_rng(cfg)
    for t in range(FULL[cfg]):
        w.standin(st, d["sigma_joint"], d["sigma_vel"])
        H.upload_state(st, bufs, env=False)
        t_next = st.t + 1
        z_root = st.pos[0, 2].copy()
        prev = None
        if bufs.prev_action is not None:
            prev = rng.normal(size=(N, w.A)).astype(np.float32)
            bufs.prev_action[:N].copy_(torch.from_numpy(prev))
        ctx.env_step_fused(bufs, with_ref_frame=(t == 0))
        w.env_step(st, prev_action=prev)
        g = H.download(bufs, N)
        if t > 0:
            g.ref_frame = st.ref_frame.copy()     # not written without the optional buffer
        live = H.compare_step(g, st, c["r_min"], c["h_term"], c["grace"], t_next, z_root, live)
        H.compare_sim_obs(g, st, live, "full-size step %d" % t)
        n_done += int((st.terminated | st.truncated).sum())
    print("cfg %d: %d resets, %d envs at reward ties" % (cfg, n_done, int((~live).sum())))
    assert live.mean() > 0.999
    assert n_done > 0


def test_full_size_policy(world):
    cfg, d, w, ctx, bufs = world
    N = d["n_envs"]
    pol = d["policy"]
    A = pol["dims"][-1]
    st = w.state(N)
    st.n[:] = (np.arange(N, dtype=np.uint64) * 2654435761 % (1 << 32)).astype(np.uint32)
    w.reset_envs(st)
    w.standin(st, d["sigma_joint"], d["sigma_vel"])
    w.env_step(st)
    bufs.obs.copy_(torch.from_numpy(st.obs))
    bufs.env_n.copy_(torch.from_numpy(st.n.view(np.int32)))
    mean = torch.empty((N, A), device="cuda")
    act = torch.empty((N, A), device="cuda")
    logp = torch.empty(N, device="cuda")
    ctx.policy_act(bufs.obs, bufs.env_n, N, mean, act, logp)
    torch.cuda.synchronize()
    gm, ga, gl = mean.cpu().numpy(), act.cpu().numpy(), logp.cpu().numpy()

    om, oa, olp = oracle.policy(pol, d["config"]["seed"], st.obs, st.n)
    tol = 2e-2 if pol["bf16"] else 1e-4
    for name, gg, oo in (("mean", gm, om), ("action", ga, oa)):
        err = np.linalg.norm(gg - oo, axis=1) / np.linalg.norm(oo, axis=1)
        assert err.max() <= tol, "%s: worst per-env relative error %.3e at env %d" % (
            name, err.max(), int(np.argmax(err)))
        print("cfg %d %s (all %d envs): max rel err %.2e" % (cfg, name, N, err.max()))
    lbad = ~(np.abs(gl - olp) <= 1e-5 * np.abs(olp) + 1e-4)
    assert not lbad.any(), "logp at envs %s" % np.flatnonzero(lbad)[:5]
    sig = np.exp(pol["log_std"].astype(np.float64))
    zg = (ga.astype(np.float64) - gm) / sig
    zo = (oa.astype(np.float64) - om) / sig
    assert np.abs(zg - zo).max() < 1e-3

    # every env: finite, logp consistent with its own noise, noise ~ N(0, 1)
    assert np.all(np.isfinite(gm)) and np.all(np.isfinite(ga)) and np.all(np.isfinite(gl))
    z = (ga.astype(np.float64) - gm) / sig
    lp = -(0.5 * z * z + np.log(sig) + 0.5 * np.log(2 * np.pi)).sum(axis=1)
    assert np.all(np.abs(lp - gl) <= 1e-4 * np.abs(lp) + 1e-2)
    zf = z.ravel()
    n = zf.size
    assert abs(zf.mean()) < 5.0 / np.sqrt(n)
    assert abs(zf.var() - 1.0) < 5.0 * np.sqrt(2.0 / n)


def test_full_size_value(world):
    """The critic at full size (large-batch GEMM tiles and the value head)
    against the oracle on every env."""
    cfg, d, w, ctx, bufs = world
    N = d["n_envs"]
    st = w.state(N)
    w.reset_envs(st)
    w.standin(st, d["sigma_joint"], d["sigma_vel"])
    w.env_step(st)
    bufs.obs.copy_(torch.from_numpy(st.obs))
    v = torch.empty(N, device="cuda")
    ctx.value(bufs.obs, N, v)
    torch.cuda.synchronize()
    gv = v.cpu().numpy()
    ov = oracle.value(d["critic"], st.obs)
    s = np.sqrt(np.mean(ov.astype(np.float64) ** 2))
    tol = 2e-2 if d["critic"]["bf16"] else 1e-4
    err = np.abs(gv - ov) / np.maximum(np.abs(ov), s)
    assert err.max() <= tol, "value: worst %.3e at env %d" % (err.max(), int(np.argmax(err)))
    print("cfg %d value (all %d envs): max rel err %.2e" % (cfg, N, err.max()))
    assert np.all(np.isfinite(gv))
