"""The rollout captured as a HIP graph (policy_act, stand-in physics,
env_step_fused for several steps) replays to bitwise the results of the same
calls run eagerly.  Every call is stream-ordered, allocates nothing and reads
nothing back, and the per-env Philox counters live in device memory, so each
replay draws fresh numbers.  Replays are checked several times, with eager
work and synchronisations in between."""
import numpy as np
import pytest
import torch

from paper_2609_09821_amd import binding, synth

pytestmark = pytest.mark.gpu

STATE = binding.EnvBuffers.SIM + binding.EnvBuffers.ENV + ("reward", "terminated", "truncated",
                                                            "obs")


def _snapshot(bufs, extra=()):
    out = {k: getattr(bufs, k).clone() for k in STATE}
    for i, t in enumerate(extra):
        out["extra%d" % i] = t.clone()
    return out


def _restore(bufs, snap, extra=()):
    for k in STATE:
        getattr(bufs, k).copy_(snap[k])
    for i, t in enumerate(extra):
        t.copy_(snap["extra%d" % i])


def _equal(a, b):
    return all(torch.equal(a[k], b[k]) for k in a)


@pytest.mark.parametrize("cfg,N", [(1, 64), (2, 1000), (3, 5000), (4, 20000), (6, 3000)])
def test_graph_replay_matches_eager(cfg, N):
    d = synth.make_world(cfg, n_envs=N)
    ctx = binding.Context(d, max_envs=N)
    bufs = ctx.buffers(N)
    A = d["policy"]["dims"][-1]
    mean = torch.zeros((N, A), device="cuda")
    act = torch.zeros((N, A), device="cuda")
    logp = torch.zeros(N, device="cuda")
    extra = (mean, act, logp)
    if bufs.prev_action is not None:
        bufs.prev_action = act               # the observation's previous action
    T = 3

    def rollout():
        for _ in range(T):
            ctx.policy_act(bufs.obs, bufs.env_n, N, mean, act, logp)
            ctx.standin_physics(bufs, d["sigma_joint"], d["sigma_vel"])
            ctx.env_step_fused(bufs, with_ref_frame=False)

    ctx.reset_envs(bufs)
    torch.cuda.synchronize()
    s0 = _snapshot(bufs, extra)
    rollout()
    torch.cuda.synchronize()
    eager1 = _snapshot(bufs, extra)
    rollout()
    torch.cuda.synchronize()
    eager2 = _snapshot(bufs, extra)
    assert not _equal(eager1, eager2)

    _restore(bufs, s0, extra)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            rollout()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    # capture runs nothing
    assert _equal(_snapshot(bufs, extra), s0)

    for rep in range(3):
        _restore(bufs, s0, extra)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert _equal(_snapshot(bufs, extra), eager1), "replay %d differs from eager" % rep
        g.replay()                       # continues from the replayed state
        torch.cuda.synchronize()
        assert _equal(_snapshot(bufs, extra), eager2), "second replay %d differs" % rep
        # unrelated eager work between replays
        torch.cuda.synchronize()
        ctx.standin_physics(bufs, d["sigma_joint"], d["sigma_vel"])
        torch.cuda.synchronize()
    del g
    ctx.close()


@pytest.mark.parametrize("cfg,N", [(2, 1000), (6, 3000)])
def test_rollout_graph_with_storage_and_gae(cfg, N):
    """A whole PPO rollout as one graph: T steps of policy, value, stand-in
    physics and env step written in place into the rollout storage, the value
    of the last observation, then GAE with the rollout summaries; replays
    match the eager run bitwise, also when continued from the replayed state."""
    T = 4
    d = synth.make_world(cfg, n_envs=N)
    ctx = binding.Context(d, max_envs=N)
    bufs = ctx.buffers(N)
    ro = binding.RolloutStorage(ctx, N, T)
    names = ("obs", "mean", "action", "logp", "value", "reward", "terminated", "truncated",
             "advantage", "ret", "ep_return", "ep_length", "summary")
    state = lambda: [getattr(bufs, k) for k in binding.EnvBuffers.SIM + binding.EnvBuffers.ENV] + \
        [getattr(ro, k) for k in names]

    def rollout():
        for t in range(T):
            ctx.policy_act(ro.obs[t], bufs.env_n, N, ro.mean[t], ro.action[t], ro.logp[t])
            ctx.value(ro.obs[t], N, ro.value[t])
            ctx.standin_physics(bufs, d["sigma_joint"], d["sigma_vel"])
            ro.env_bufs(bufs, t)
            ctx.env_step_fused(bufs, with_ref_frame=False)
        ctx.value(ro.obs[T], N, ro.value[T])
        ctx.gae(ro, synth.GAMMA, synth.LAMBDA)
        # the last observation starts the next rollout
        ro.obs[0].copy_(ro.obs[T])

    bufs.obs = ro.obs[0]
    ctx.reset_envs(bufs)
    torch.cuda.synchronize()
    s0 = [x.clone() for x in state()]
    rollout()
    torch.cuda.synchronize()
    eager1 = [x.clone() for x in state()]
    rollout()
    torch.cuda.synchronize()
    eager2 = [x.clone() for x in state()]
    assert not all(torch.equal(a, b) for a, b in zip(eager1, eager2))
    assert eager1[-1][3].item() > 0 or cfg == 6   # episodes ended (w6: grace period)

    def restore(snap):
        for dst, src in zip(state(), snap):
            dst.copy_(src)

    restore(s0)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            rollout()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    assert all(torch.equal(a, b) for a, b in zip(state(), s0)), "capture ran work"
    for rep in range(3):
        restore(s0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k, (a, b) in enumerate(zip(state(), eager1)):
            assert torch.equal(a, b), "replay %d differs from eager in buffer %d" % (rep, k)
        g.replay()
        torch.cuda.synchronize()
        for k, (a, b) in enumerate(zip(state(), eager2)):
            assert torch.equal(a, b), "second replay %d differs in buffer %d" % (rep, k)
        ctx.standin_physics(bufs, d["sigma_joint"], d["sigma_vel"])
        torch.cuda.synchronize()
    del g
    ctx.close()
