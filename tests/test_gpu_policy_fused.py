"""The one-launch bf16 policy and critic (every layer in one kernel, the
activations held in LDS between layers, weights read in MFMA fragment order)
against the oracle on every env.

Cases cover the widths and depths the kernel takes: hidden layers of 256,
512, 768 and 1024 features (one to four MFMA tiles per wave), 32 to 128
padded actions, one layer (no hidden layer) up to eight, an observation 961
wide (1024 padded: the widest LDS row), a single env, ragged last blocks of
64 envs and a full grid of 16384 envs.  Policies it does not hold (a
1280-wide hidden layer, nine layers) take the per-layer kernels, checked the
same way.  The critic variant (hidden layers, then the fp32 value head)
runs over the same widths and depths.  Tolerances as in the full-size parity
test.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_09821_amd import binding, synth
from tests.worlds import clip_from_arrays, custom_world

pytestmark = pytest.mark.gpu

CHAIN6 = list(range(-1, 5))                  # observation 91 wide
# a root and seven chains of nine bodies: 64 bodies, observation 961 wide
COMB64 = [-1] + [0 if j == 0 else 9 * b + j for b in range(7) for j in range(9)]


def _world(parent, hidden, A, seed, critic_hidden=None):
    B = len(parent)
    d = custom_world(parent, [0] + [1] * (B - 1), [[0, 0, 0]] + [[0.1, 0, 0]] * (B - 1), [1.0] * B,
                     [clip_from_arrays(np.zeros((2, 3)), np.tile([1, 0, 0, 0], (2, 1)),
                                       np.tile([1, 0, 0, 0], (2, B - 1, 1)))])
    D = 15 * B + 1
    d["policy"] = synth.make_policy(np.random.default_rng(seed), [D] + list(hidden) + [A], True)
    if critic_hidden is not None:
        d["critic"] = synth.make_policy(np.random.default_rng(seed + 1), [D] + list(critic_hidden) + [1],
                                        True)
    return d


def check_policy(d, N):
    """policy_act on N envs of random observations against the oracle."""
    pol = d["policy"]
    D, A = pol["dims"][0], pol["dims"][-1]
    d["n_envs"] = N
    print("policy %s at %d envs" % (pol["dims"], N), flush=True)
    ctx = binding.Context(d, max_envs=N, critic=False)
    assert ctx.info.obs_dim == D
    rng = np.random.default_rng(N + D)
    obs = rng.normal(size=(D, N)).astype(np.float32)
    n = rng.integers(0, 1 << 32, size=N, dtype=np.uint64).astype(np.uint32)
    mean = torch.empty((N, A), device="cuda")
    act = torch.empty((N, A), device="cuda")
    logp = torch.empty(N, device="cuda")
    ctx.policy_act(torch.from_numpy(obs).cuda(), torch.from_numpy(n.view(np.int32)).cuda(), N,
                   mean, act, logp)
    torch.cuda.synchronize()
    gm, ga, gl = mean.cpu().numpy(), act.cpu().numpy(), logp.cpu().numpy()
    ctx.close()
    om, oa, olp = oracle.policy(pol, d["config"]["seed"], obs, n)
    for name, gg, oo in (("mean", gm, om), ("action", ga, oa)):
        err = np.linalg.norm(gg - oo, axis=1) / np.linalg.norm(oo, axis=1)
        assert err.max() <= 2e-2, "%s: worst per-env relative error %.3e at env %d" % (
            name, err.max(), int(np.argmax(err)))
        print("%s (all %d envs): max rel err %.2e" % (name, N, err.max()))
    lbad = ~(np.abs(gl - olp) <= 1e-5 * np.abs(olp) + 1e-4)
    assert not lbad.any(), "logp at envs %s" % np.flatnonzero(lbad)[:5]
    assert np.all(np.isfinite(gm)) and np.all(np.isfinite(ga))


@pytest.mark.parametrize("parent,hidden,A,N", [
    (CHAIN6, [256, 768], 8, 1300),        # one and three tiles per wave, one action tile
    (CHAIN6, [1024, 512], 100, 16384),    # four and two tiles per wave, four action tiles
    (CHAIN6, [512, 1024], 40, 1),         # a single env
    (CHAIN6, [], 64, 200),                # no hidden layer
    (CHAIN6, [256] * 7, 8, 130),          # eight layers
    (COMB64, [1024], 69, 333),            # 1024-wide padded observation, three action tiles
    (CHAIN6, [512], 96, 777),             # three full action tiles
    (CHAIN6, [256], 128, 300),            # the widest action set: four full tiles
], ids=["256-768", "1024-512-full-grid", "one-env", "one-layer", "eight-layers", "obs-961",
        "96-actions", "128-actions"])
def test_fused_policy_shapes(parent, hidden, A, N):
    check_policy(_world(parent, hidden, A, 5), N)


@pytest.mark.parametrize("hidden,N", [([1280], 700), ([256] * 8, 130)],
                         ids=["hidden-1280", "nine-layers"])
def test_policies_outside_the_fused_kernel(hidden, N):
    check_policy(_world(CHAIN6, hidden, 8, 6), N)


def check_value(d, N):
    """value on N envs of random observations against the oracle."""
    crit = d["critic"]
    D = crit["dims"][0]
    d["n_envs"] = N
    print("critic %s at %d envs" % (crit["dims"], N), flush=True)
    ctx = binding.Context(d, max_envs=N)
    obs = np.random.default_rng(N + 7).normal(size=(D, N)).astype(np.float32)
    v = torch.empty(N, device="cuda")
    ctx.value(torch.from_numpy(obs).cuda(), N, v)
    torch.cuda.synchronize()
    gv = v.cpu().numpy()
    ctx.close()
    ov = oracle.value(crit, obs)
    s = np.sqrt(np.mean(ov.astype(np.float64) ** 2))
    err = np.abs(gv - ov) / np.maximum(np.abs(ov), s)
    assert err.max() <= 2e-2, "value: worst %.3e at env %d" % (err.max(), int(np.argmax(err)))
    print("value (all %d envs): max rel err %.2e" % (N, err.max()))
    assert np.all(np.isfinite(gv))


@pytest.mark.parametrize("parent,hidden,N", [
    (CHAIN6, [256, 768], 1300),
    (CHAIN6, [1024, 512], 16384),
    (CHAIN6, [512], 1),
    (CHAIN6, [256] * 8, 130),             # eight hidden layers
    (COMB64, [1024, 256], 333),           # 1024-wide padded observation
    (CHAIN6, [1280], 700),                # too wide: per-layer kernels
], ids=["256-768", "1024-512-full-grid", "one-env", "eight-hidden", "obs-961", "hidden-1280"])
def test_fused_critic_shapes(parent, hidden, N):
    check_value(_world(parent, [256], 8, 9, critic_hidden=hidden), N)
