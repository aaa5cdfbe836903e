"""The persistent bf16 GEMM of large batches at the edges of its schedule,
against the oracle on every env, through the hidden layers of a critic whose
1280-wide first layer the one-launch kernel does not hold (the policy with
the other two widths runs in the one-launch kernel, checked too).

A six-body chain has a 91-wide observation, whose first layer then runs two K
steps per tile (the shortest pipeline: the next tile's loads and biases are
staged while the current tile is one step from done).  The hidden widths give
one, two, three and five feature blocks per env block; the env counts leave
ragged last tiles and, at 16684 envs, fewer tiles than compute units (one
tile per workgroup).  Tolerances as in the full-size parity test.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_09821_amd import binding, synth
from tests.worlds import clip_from_arrays, custom_world

pytestmark = pytest.mark.gpu


def _chain_world(dims):
    B = 6
    d = custom_world(list(range(-1, B - 1)), [0] + [1] * (B - 1),
                     [[0, 0, 0]] + [[0.1, 0, 0]] * (B - 1), [1.0] * B,
                     [clip_from_arrays(np.zeros((2, 3)), np.tile([1, 0, 0, 0], (2, 1)),
                                       np.tile([1, 0, 0, 0], (2, B - 1, 1)))])
    d["policy"] = synth.make_policy(np.random.default_rng(3), dims, True)
    d["critic"] = synth.make_policy(np.random.default_rng(4), [dims[0], 1280] + dims[1:-1] + [1], True)
    return d


@pytest.mark.parametrize("hidden,N", [((256, 512), 16384 + 300), ((768, 256), 65536 + 44)])
def test_persistent_gemm_schedule_edges(hidden, N):
    A = 8
    D = 91
    dims = [D, hidden[0], hidden[1], A]
    d = _chain_world(dims)
    d["n_envs"] = N
    print("gemm shapes %s at %d envs" % (dims, N), flush=True)
    ctx = binding.Context(d, max_envs=N)
    assert ctx.info.obs_dim == D
    rng = np.random.default_rng(N)
    obs = rng.normal(size=(D, N)).astype(np.float32)
    n = rng.integers(0, 1 << 32, size=N, dtype=np.uint64).astype(np.uint32)
    mean = torch.empty((N, A), device="cuda")
    act = torch.empty((N, A), device="cuda")
    logp = torch.empty(N, device="cuda")
    ctx.policy_act(torch.from_numpy(obs).cuda(), torch.from_numpy(n.view(np.int32)).cuda(), N,
                   mean, act, logp)
    v = torch.empty(N, device="cuda")
    ctx.value(torch.from_numpy(obs).cuda(), N, v)
    torch.cuda.synchronize()
    gm, ga, gl = mean.cpu().numpy(), act.cpu().numpy(), logp.cpu().numpy()
    gv = v.cpu().numpy()
    ctx.close()

    ov = oracle.value(d["critic"], obs)
    sv = np.sqrt(np.mean(ov.astype(np.float64) ** 2))
    verr = np.abs(gv - ov) / np.maximum(np.abs(ov), sv)
    assert verr.max() <= 2e-2, "value: worst %.3e at env %d" % (verr.max(), int(np.argmax(verr)))
    print("value (all %d envs): max rel err %.2e" % (N, verr.max()))

    pol = d["policy"]
    om, oa, olp = oracle.policy(pol, d["config"]["seed"], obs, n)
    for name, gg, oo in (("mean", gm, om), ("action", ga, oa)):
        err = np.linalg.norm(gg - oo, axis=1) / np.linalg.norm(oo, axis=1)
        assert err.max() <= 2e-2, "%s: worst per-env relative error %.3e at env %d" % (
            name, err.max(), int(np.argmax(err)))
        print("%s (all %d envs): max rel err %.2e" % (name, N, err.max()))
    lbad = ~(np.abs(gl - olp) <= 1e-5 * np.abs(olp) + 1e-4)
    assert not lbad.any(), "logp at envs %s" % np.flatnonzero(lbad)[:5]
    assert np.all(np.isfinite(gm)) and np.all(np.isfinite(ga))
