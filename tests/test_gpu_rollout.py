"""The rollout end on the GPU against the oracle: value head, GAE with the
rollout summaries, and a whole teacher-forced rollout written in place into
the rollout storage (Fig. 3: storage.write of every step).

Tolerances (besides those of gpu_helpers):
* value: |g - o| <= tol * max(|o|, s), s = RMS of the oracle's values over
  the batch, tol = 2e-2 for bf16 critics, 1e-4 for fp32 (the policy's
  per-env tolerances applied to a scalar output);
* advantages and returns: |g - o| <= 2e-6 max(|o|, 1) (both float64 inside,
  stored as float32: at most a rounding of the final conversion apart);
* summaries: counts exact; float64 sums |g - o| <= 1e-9 max(|o|, 1);
* running-episode accumulators: bit-exact (float32 adds in step order).
"""
import ctypes as C

import numpy as np
import pytest
import torch

import oracle
from paper_2609_09821_amd import binding, synth
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu

SUM = {k: i for i, k in enumerate(binding.SUMMARY_FIELDS)}


def value_close(g, o, bf16, what=""):
    g = np.asarray(g, np.float64)
    o = np.asarray(o, np.float64)
    s = np.sqrt(np.mean(o * o))
    tol = 2e-2 if bf16 else 1e-4
    err = np.abs(g - o) / np.maximum(np.abs(o), s)
    assert err.max() <= tol, "%s value: worst relative error %.3e at %d" % (what, err.max(),
                                                                          int(err.argmax()))
    return err.max()


def _obs_batch(w, d, N, steps=1):
    st = w.state(N)
    st.n[:] = (np.arange(N, dtype=np.uint64) * 2654435761 % (1 << 32)).astype(np.uint32)
    w.reset_envs(st)
    for _ in range(steps):
        w.standin(st, d["sigma_joint"], d["sigma_vel"])
        w.env_step(st)
    return st.obs


# ---------------------------------------------------------------- value head
@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 6])
def test_value_parity(cfg):
    N = {1: 64, 2: 1000, 3: 1300, 4: 700, 6: 900}[cfg]
    d = synth.make_world(cfg, n_envs=N)
    w = oracle.World(d)
    ctx = binding.Context(d, max_envs=N)
    obs = _obs_batch(w, d, N)
    go = torch.from_numpy(obs).cuda()
    v = torch.full((N,), -7.0, device="cuda")
    ctx.value(go, N, v)
    torch.cuda.synchronize()
    ov = oracle.value(d["critic"], obs)
    err = value_close(v.cpu().numpy(), ov, d["critic"]["bf16"], "cfg %d" % cfg)
    print("cfg %d value: max rel err %.2e" % (cfg, err))
    ctx.close()


@pytest.mark.parametrize("bf16", [False, True])
def test_one_layer_and_replaced_critic(bf16):
    # a linear critic (the head reads the observation itself), then a
    # replacement by the workload's MLP critic on the same context
    cfg = 3 if bf16 else 2
    N = 777
    d = synth.make_world(cfg, n_envs=N)
    w = oracle.World(d)
    ctx = binding.Context(d, max_envs=N, critic=False)
    obs = _obs_batch(w, d, N)
    go = torch.from_numpy(obs).cuda()
    v = torch.zeros(N, device="cuda")
    with pytest.raises(binding.ImError, match="no critic"):
        ctx.value(go, N, v)
    D = d["policy"]["dims"][0]
    rng = np.random.default_rng(11)
    Wl = (rng.uniform(-1, 1, size=(1, D)) / np.sqrt(D)).astype(np.float32)
    if bf16:
        Wl = synth.bf16_round(Wl)
    lin = dict(dims=[D, 1], bf16=bf16, W=[Wl], b=[np.array([0.125], np.float32)],
               log_std=None)
    desc = binding.Description(d)
    binding.im_set_critic(ctx.ptr, desc._mlp(lin))
    ctx.value(go, N, v)
    torch.cuda.synchronize()
    value_close(v.cpu().numpy(), oracle.value(lin, obs), bf16, "linear")
    binding.im_set_critic(ctx.ptr, desc._mlp(d["critic"]))
    ctx.value(go, N, v)
    torch.cuda.synchronize()
    value_close(v.cpu().numpy(), oracle.value(d["critic"], obs), bf16, "replaced")
    ctx.close()


def test_critic_validation():
    d = synth.make_world(2, n_envs=64)
    ctx = binding.Context(d, max_envs=64, critic=False)
    desc = binding.Description(d)
    crit = d["critic"]
    bad = [
        (dict(crit, dims=[crit["dims"][0] + 1] + crit["dims"][1:]), "observation width"),
        (dict(crit, dims=crit["dims"][:-1] + [2]), "output width"),
        (dict(crit, bf16=True), "dtype"),
    ]
    for net, words in bad:
        with pytest.raises(binding.ImError, match=words):
            binding.im_set_critic(ctx.ptr, desc._mlp(net))
    ctx.close()


# ----------------------------------------------------------------------- GAE
def _upload(x, ld=None):
    T, N = x["reward"].shape
    ld = ld or N

    def dev(a, rows, dtype):
        t = torch.full((rows, ld), 99, dtype=dtype, device="cuda")
        t[:, :N] = torch.from_numpy(np.ascontiguousarray(a))
        return t

    class R:
        pass
    r = R()
    r.T, r.n_envs, r.ld = T, N, ld
    r.reward = dev(x["reward"], T, torch.float32)
    r.terminated = dev(x["term"], T, torch.uint8)
    r.truncated = dev(x["trunc"], T, torch.uint8)
    r.value = dev(x["value"], T + 1, torch.float32)
    r.advantage = torch.full((T, ld), -5.0, device="cuda")
    r.ret = torch.full((T, ld), -5.0, device="cuda")
    r.ep_return = torch.full((ld,), -1.0, device="cuda")
    r.ep_return[:N] = torch.from_numpy(x["ep_return"])
    r.ep_length = torch.full((ld,), -1, dtype=torch.int32, device="cuda")
    r.ep_length[:N] = torch.from_numpy(x["ep_length"])
    r.summary = torch.full((len(SUM),), -3.0, dtype=torch.float64, device="cuda")
    r.struct = lambda g, l, s=True: binding.RolloutStorage.struct(r, g, l, s)
    return r


def _check_gae(r, x, gamma, lam, summary=True):
    N = r.n_envs
    # the call takes gamma and lambda as float32: the oracle gets the same numbers
    gamma, lam = float(np.float32(gamma)), float(np.float32(lam))
    oa, orr = oracle.gae(x["reward"], x["term"], x["trunc"], x["value"], gamma, lam)
    torch.cuda.synchronize()
    ga = r.advantage[:, :N].cpu().numpy()
    gr = r.ret[:, :N].cpu().numpy()
    for name, g, o in (("advantage", ga, oa), ("return", gr, orr)):
        err = np.abs(g.astype(np.float64) - o) / np.maximum(np.abs(o), 1.0)
        assert err.max() <= 2e-6, "%s: worst %.3e" % (name, err.max())
    if not summary:
        return
    os_, oepr, oepl = oracle.rollout_summary(x["reward"], x["term"], x["trunc"], x["value"], oa,
                                             orr, x["ep_return"], x["ep_length"])
    gs = r.summary.cpu().numpy()
    for k in ("n_terminated", "n_truncated", "n_episodes", "episode_length_sum"):
        assert gs[SUM[k]] == os_[SUM[k]], k
    err = np.abs(gs - os_) / np.maximum(np.abs(os_), 1.0)
    assert err.max() <= 1e-9, "summary field %s: %.3e" % (binding.SUMMARY_FIELDS[err.argmax()],
                                                          err.max())
    assert np.array_equal(r.ep_return[:N].cpu().numpy(), oepr)
    assert np.array_equal(r.ep_length[:N].cpu().numpy(), oepl)


@pytest.mark.parametrize("T,N,seed", [(32, 3000, 1), (1, 700, 2), (8, 257, 3)])
def test_gae_and_summary_parity(T, N, seed):
    d = synth.make_world(2, n_envs=max(N, 1))
    ctx = binding.Context(d, max_envs=max(N, 1), critic=False)
    x = synth.rollout_inputs(seed, T, N)
    r = _upload(x)
    ctx.gae(r, synth.GAMMA, synth.LAMBDA)
    _check_gae(r, x, synth.GAMMA, synth.LAMBDA)
    ctx.close()


def test_gae_leading_dimension_tail_and_no_summary():
    T, N, ld = 12, 1000, 1000 + 77
    d = synth.make_world(2, n_envs=N)
    ctx = binding.Context(d, max_envs=N, critic=False)
    x = synth.rollout_inputs(4, T, N, p_term=0.1, p_trunc=0.05)
    r = _upload(x, ld)
    ctx.gae(r, 0.98, 0.99, summary=False)
    _check_gae(r, x, 0.98, 0.99, summary=False)
    assert (r.advantage[:, N:] == -5.0).all() and (r.ret[:, N:] == -5.0).all()
    # without summaries the running-episode accumulators are not touched
    assert (r.ep_return[:N].cpu().numpy() == x["ep_return"]).all()
    assert (r.summary == -3.0).all()
    ctx.gae(r, 0.98, 0.99)
    _check_gae(r, x, 0.98, 0.99)
    assert (r.ep_return[N:] == -1.0).all() and (r.ep_length[N:] == -1).all()
    ctx.close()


def test_gae_zero_envs_and_bad_arguments():
    d = synth.make_world(2, n_envs=64)
    ctx = binding.Context(d, max_envs=64, critic=False)
    x = synth.rollout_inputs(5, 4, 64)
    r = _upload(x)
    r.n_envs = 0
    ctx.gae(r, synth.GAMMA, synth.LAMBDA)
    torch.cuda.synchronize()
    assert (r.summary == 0).all() and (r.advantage == -5.0).all()
    r.n_envs = 64
    for field, val, words in (("T", 0, "T must"), ("gamma", 1.5, "gamma"), ("n_envs", 65, "n_envs")):
        s = r.struct(synth.GAMMA, synth.LAMBDA)
        setattr(s, field, val)
        with pytest.raises(binding.ImError, match=words):
            binding.im_gae(ctx.ptr, s, binding._stream(None))
    s = r.struct(synth.GAMMA, synth.LAMBDA)
    s.ep_return = None
    with pytest.raises(binding.ImError, match="ep_return"):
        binding.im_gae(ctx.ptr, s, binding._stream(None))
    ctx.close()


# ------------------------------------------------- rollout into the storage
@pytest.mark.parametrize("cfg,N", [(2, 600), (6, 500)])
def test_rollout_written_in_place(cfg, N):
    """T teacher-forced steps with every output pointed at its storage slot:
    slot t holds the step's policy outputs and value (on the observation of
    slot t) and its reward and flags, slot t + 1 the post-step observation."""
    T = 6
    d = synth.make_world(cfg, n_envs=N)
    c = d["config"]
    w = oracle.World(d)
    ctx = binding.Context(d, max_envs=N)
    bufs = ctx.buffers(N)
    ro = binding.RolloutStorage(ctx, N, T)
    pol, crit = d["policy"], d["critic"]
    bf16 = pol["bf16"]
    A = pol["dims"][-1]
    D0 = w.D - (A if c["obs_prev_action"] else 0)    # rows before the previous action
    st = w.state(N)
    w.reset_envs(st)
    H.upload_state(st, bufs)
    bufs.obs = ro.obs[0]
    ctx.reset_envs(bufs)
    live = np.ones(N, bool)
    ovals = []
    for t in range(T):
        # GPU: policy and value on slot t, physics stand-in, env step into the slots
        ctx.policy_act(ro.obs[t], bufs.env_n, N, ro.mean[t], ro.action[t], ro.logp[t])
        ctx.value(ro.obs[t], N, ro.value[t])
        om, oa, olp = oracle.policy(pol, c["seed"], st.obs, st.n)
        ovals.append(oracle.value(crit, st.obs))
        w.standin(st, d["sigma_joint"], d["sigma_vel"])
        H.upload_state(st, bufs, env=False)
        ro.env_bufs(bufs, t)
        t_next = st.t + 1
        z_root = st.pos[0, 2].copy()
        ctx.env_step_fused(bufs)
        w.env_step(st, prev_action=oa if c["obs_prev_action"] else None)
        torch.cuda.synchronize()
        g = H.download(bufs, N)
        live = H.compare_step(g, st, c["r_min"], c["h_term"], c["grace"], t_next, z_root, live)
        gobs = ro.obs[t + 1].cpu().numpy()
        H.assert_close(gobs[:D0, live], st.obs[:D0, live], what="obs slot %d" % (t + 1))
        # policy outputs and value of slot t
        tol = 2e-2 if bf16 else 1e-4
        for name, gg, oo in (("mean", ro.mean[t].cpu().numpy(), om),
                             ("action", ro.action[t].cpu().numpy(), oa)):
            err = np.linalg.norm(gg[live] - oo[live], axis=1) / np.linalg.norm(oo[live], axis=1)
            assert err.max() <= tol, "%s slot %d: %.3e" % (name, t, err.max())
        if c["obs_prev_action"]:
            # the observation's previous action is the step's own (GPU) action,
            # zero for the envs the step reset
            done = (g.terminated | g.truncated).astype(bool)
            ga = ro.action[t].cpu().numpy()
            assert np.array_equal(gobs[D0:, ~done], ga[~done].T)
            assert (gobs[D0:, done] == 0).all()
        value_close(ro.value[t].cpu().numpy()[live], ovals[-1][live], bf16, "slot %d" % t)
        assert np.array_equal(ro.reward[t].cpu().numpy(), g.reward)
        assert np.array_equal(ro.terminated[t].cpu().numpy(), g.terminated)
    ctx.value(ro.obs[T], N, ro.value[T])
    torch.cuda.synchronize()
    value_close(ro.value[T].cpu().numpy()[live], oracle.value(crit, st.obs)[live], bf16, "slot T")
    ctx.gae(ro, synth.GAMMA, synth.LAMBDA)
    torch.cuda.synchronize()
    # every stored advantage satisfies the recursion on the stored values
    a = ro.advantage.cpu().numpy().astype(np.float64)
    V = ro.value.cpu().numpy().astype(np.float64)
    r = ro.reward.cpu().numpy().astype(np.float64)
    te = ro.terminated.cpu().numpy().astype(bool)
    dn = te | ro.truncated.cpu().numpy().astype(bool)
    nxt = np.where(te, 0.0, np.where(dn, V[:T], V[1:]))
    nxt_a = np.vstack([a[1:], np.zeros((1, N))])
    rhs = r + synth.GAMMA * nxt - V[:T] + synth.GAMMA * synth.LAMBDA * np.where(dn, 0.0, nxt_a)
    assert np.all(np.abs(a - rhs) <= 1e-5 * np.maximum(np.abs(rhs), 1.0))
    s = ro.summary.cpu().numpy()
    assert s[SUM["n_terminated"]] == te.sum() and s[SUM["n_episodes"]] == dn.sum()
    ctx.close()


# ------------------------------------------------- policy and value in one call
def _gpu_obs(ctx, d, N, steps):
    bufs = ctx.buffers(N)
    ctx.reset_envs(bufs)
    for _ in range(steps):
        ctx.standin_physics(bufs, d["sigma_joint"], d["sigma_vel"])
        ctx.env_step_fused(bufs)
    return bufs.obs.clone(), bufs.env_n.clone()


@pytest.mark.parametrize("cfg,N", [(2, 1000), (3, 1300), (4, 20000), (5, 17000)])
def test_policy_act_value_equals_separate_calls(cfg, N):
    """One call of both networks gives the bits of the two calls made apart,
    also right after a call on another observation (the staged observation
    is always this call's own)."""
    print("policy_act_value cfg %d N %d" % (cfg, N), flush=True)
    d = synth.make_world(cfg, n_envs=N)
    ctx = binding.Context(d, max_envs=N)
    A = d["policy"]["dims"][-1]
    obs1, n1 = _gpu_obs(ctx, d, N, 1)
    obs2, n2 = _gpu_obs(ctx, d, N, 3)

    def outs():
        return (torch.full((N, A), -9.0, device="cuda"), torch.full((N, A), -9.0, device="cuda"),
                torch.full((N,), -9.0, device="cuda"), torch.full((N,), -9.0, device="cuda"))

    def separate(obs, n):
        m, a, lp, v = outs()
        ctx.policy_act(obs, n, N, m, a, lp)
        ctx.value(obs, N, v)
        return m, a, lp, v

    def combined(obs, n):
        m, a, lp, v = outs()
        ctx.policy_act_value(obs, n, N, m, a, lp, v)
        return m, a, lp, v

    ref1 = separate(obs1, n1)
    got2 = combined(obs2, n2)
    ref2 = separate(obs2, n2)
    got1 = combined(obs1, n1)
    torch.cuda.synchronize()
    for got, ref in ((got1, ref1), (got2, ref2)):
        for name, g, r in zip(("mean", "action", "logp", "value"), got, ref):
            assert torch.equal(g, r), "%s differs from the separate calls" % name
    assert not torch.equal(ref1[3], ref2[3])


@pytest.mark.parametrize("wide", ["both", "critic"])
def test_policy_act_value_per_layer_networks(wide):
    """Networks beyond the one-launch kernel (a 1280-wide first hidden layer)
    at a large bf16 batch: with both per-layer, the critic's first layer reads
    the observation the policy staged; with the policy in one launch the critic
    stages its own.  Either way the bits of the two separate calls."""
    N = 16384 + 700
    print("policy_act_value per-layer %s N %d" % (wide, N), flush=True)
    d = synth.make_world(4, n_envs=N)
    D, A = d["policy"]["dims"][0], d["policy"]["dims"][-1]
    if wide == "both":
        d["policy"] = synth.make_policy(np.random.default_rng(11), [D, 1280, 512, A], True)
    d["critic"] = synth.make_policy(np.random.default_rng(12), [D, 1280, 512, 1], True)
    ctx = binding.Context(d, max_envs=N)
    obs1, n1 = _gpu_obs(ctx, d, N, 1)
    obs2, n2 = _gpu_obs(ctx, d, N, 2)
    res = {}
    for key, obs, n, comb in (("s1", obs1, n1, False), ("c2", obs2, n2, True),
                              ("s2", obs2, n2, False), ("c1", obs1, n1, True)):
        m = torch.full((N, A), -9.0, device="cuda")
        a = torch.full((N, A), -9.0, device="cuda")
        lp = torch.full((N,), -9.0, device="cuda")
        v = torch.full((N,), -9.0, device="cuda")
        if comb:
            ctx.policy_act_value(obs, n, N, m, a, lp, v)
        else:
            ctx.policy_act(obs, n, N, m, a, lp)
            ctx.value(obs, N, v)
        res[key] = (m, a, lp, v)
    torch.cuda.synchronize()
    for c, s_ in (("c1", "s1"), ("c2", "s2")):
        for name, g, r in zip(("mean", "action", "logp", "value"), res[c], res[s_]):
            assert torch.equal(g, r), "%s differs from the separate calls" % name
    assert not torch.equal(res["s1"][3], res["s2"][3])
    # and the value is the critic's, against the oracle on sampled envs
    idx = np.random.default_rng(5).choice(N, 64, replace=False)
    ob = obs1.cpu().numpy()[:, idx].astype(np.float32)
    ov = oracle.value(d["critic"], ob)
    gv = res["c1"][3].cpu().numpy()[idx]
    sv = np.sqrt(np.mean(ov.astype(np.float64) ** 2))
    assert np.max(np.abs(gv - ov) / np.maximum(np.abs(ov), sv)) <= 2e-2
    ctx.close()


def test_policy_act_value_errors_before_any_launch():
    """Without a critic, or with a null value buffer, the combined call fails
    with the two calls' errors and writes nothing."""
    d = synth.make_world(2, n_envs=64)
    N, A = 64, d["policy"]["dims"][-1]
    obs, env_n = None, None
    for critic in (False, True):
        ctx = binding.Context(d, max_envs=N, critic=critic)
        bufs = ctx.buffers(N)
        ctx.reset_envs(bufs)
        obs, env_n = bufs.obs, bufs.env_n
        m = torch.full((N, A), -9.0, device="cuda")
        a = torch.full((N, A), -9.0, device="cuda")
        lp = torch.full((N,), -9.0, device="cuda")
        v = torch.full((N,), -9.0, device="cuda")
        if not critic:
            with pytest.raises(binding.ImError, match="critic"):
                ctx.policy_act_value(obs, env_n, N, m, a, lp, v)
        else:
            with pytest.raises(binding.ImError, match="NULL buffer"):
                binding.im_policy_act_value(ctx.ptr, obs.data_ptr(), obs.shape[1], env_n.data_ptr(), N,
                                            m.data_ptr(), a.data_ptr(), lp.data_ptr(), None)
            with pytest.raises(binding.ImError, match="n_envs"):
                ctx.policy_act_value(obs, env_n, N + 1, m, a, lp, v)
        torch.cuda.synchronize()
        assert bool((m == -9.0).all()) and bool((v == -9.0).all())
        ctx.close()
