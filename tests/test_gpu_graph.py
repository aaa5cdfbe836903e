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
