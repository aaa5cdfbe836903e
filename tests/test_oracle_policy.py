"""Pins of the oracle policy against torch's CPU linear layers and distributions."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_09821_amd import synth


def _torch_mean(pol, obs, bf16):
    h = torch.tensor(obs.T.astype(np.float64))
    rnd = (lambda x: x.to(torch.bfloat16).to(torch.float64)) if bf16 else (lambda x: x)
    h = rnd(h)
    L = len(pol["W"])
    for i, (W, b) in enumerate(zip(pol["W"], pol["b"])):
        h = torch.nn.functional.linear(h, torch.tensor(W, dtype=torch.float64),
                                       torch.tensor(b, dtype=torch.float64))
        if i < L - 1:
            h = rnd(torch.relu(h))
    return h.numpy()


@pytest.mark.parametrize("cfg", [2, 4])
def test_mean_matches_torch_linear(cfg):
    d = synth.make_world(cfg, n_envs=16)
    pol = d["policy"]
    D = pol["dims"][0]
    obs = np.random.default_rng(cfg).normal(size=(D, 16)).astype(np.float32)
    mean, action, logp = oracle.policy(pol, 1, obs, np.zeros(16, np.uint32))
    ref = _torch_mean(pol, obs, pol["bf16"])
    if pol["bf16"]:
        # torch rounds double -> bf16 through float; a double rounding flips a rare
        # hidden value by one bf16 ulp, so compare loosely
        np.testing.assert_allclose(mean, ref, rtol=0, atol=2e-3)
    else:
        np.testing.assert_allclose(mean, ref.astype(np.float32), rtol=1e-6, atol=1e-7)


def test_bf16_round_matches_torch():
    xs = np.random.default_rng(3).normal(size=5000) * 10.0 ** np.random.default_rng(4).integers(-8, 8, 5000)
    xs = xs.astype(np.float32).astype(np.float64)  # float-valued: no double rounding
    got = np.array([oracle.round_bf16(x) for x in xs])
    ref = torch.tensor(xs, dtype=torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(got, ref)


def test_actions_and_logp():
    d = synth.make_world(2, n_envs=2000)
    pol = d["policy"]
    D = pol["dims"][0]
    N = 2000
    obs = np.random.default_rng(9).normal(size=(D, N)).astype(np.float32)
    env_n = np.arange(N, dtype=np.uint32)
    mean, action, logp = oracle.policy(pol, d["config"]["seed"], obs, env_n)
    sig = np.exp(pol["log_std"].astype(np.float64))
    z = (action.astype(np.float64) - mean) / sig
    assert abs(z.mean()) < 0.01 and abs(z.std() - 1) < 0.01
    dist = torch.distributions.Normal(torch.tensor(mean, dtype=torch.float64),
                                      torch.tensor(sig, dtype=torch.float64))
    lp = dist.log_prob(torch.tensor(action, dtype=torch.float64)).sum(-1).numpy()
    np.testing.assert_allclose(logp, lp, rtol=1e-4, atol=1e-3)
    # the noise of env e, block j comes from Philox (e, n, j, tag 0)
    A = pol["dims"][-1]
    for e in (0, 17, 1999):
        for j in range((A + 3) // 4):
            zz = oracle.normals(d["config"]["seed"], e, int(env_n[e]), j, 0)
            for q in range(4):
                if 4 * j + q < A:
                    assert abs(z[e, 4 * j + q] - zz[q]) < 2e-4 * (1 + abs(zz[q]))


def test_zero_sigma_gives_mean():
    d = synth.make_world(2, n_envs=8)
    pol = dict(d["policy"])
    pol["log_std"] = np.full_like(pol["log_std"], -200.0)
    D = pol["dims"][0]
    obs = np.random.default_rng(2).normal(size=(D, 8)).astype(np.float32)
    mean, action, _ = oracle.policy(pol, 5, obs, np.zeros(8, np.uint32))
    np.testing.assert_array_equal(mean, action)
