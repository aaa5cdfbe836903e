"""im_gae_noalloc (GAE and rollout summaries without a context, the per-block
sums in the library's fixed device scratch) against im_gae on the same
rollout storage: advantages, returns, summaries and the running-episode
accumulators bit for bit (the same kernels and reduction order), on two calls
in a row, the second on a smaller rollout, so that what the first call left
in the shared scratch must not leak into the second; then the size limit."""
import numpy as np
import pytest
import torch

from paper_2609_09821_amd import binding, synth
from tests.test_gpu_rollout import _upload

pytestmark = pytest.mark.gpu

OUT = ("advantage", "ret", "summary", "ep_return", "ep_length")


def _pair(T, N, seed, ld=None):
    x = synth.rollout_inputs(seed, T, N, p_term=0.05, p_trunc=0.02)
    return _upload(x, ld), _upload(x, ld)


def test_gae_noalloc_equals_gae_on_two_calls():
    d = synth.make_world(2, n_envs=64)
    for T, N, ld, seed in ((32, 5000, 5000 + 40, 11), (7, 1300, None, 12)):
        print("gae_noalloc: T %d, %d envs" % (T, N), flush=True)
        a, b = _pair(T, N, seed, ld)
        ctx = binding.Context(d, max_envs=N, critic=False)
        ctx.gae(a, synth.GAMMA, synth.LAMBDA)
        ctx.close()
        binding.gae_noalloc(b, synth.GAMMA, synth.LAMBDA)
        torch.cuda.synchronize()
        for k in OUT:
            assert torch.equal(getattr(a, k), getattr(b, k)), "%s differs (T %d, N %d)" % (k, T, N)
        assert int(b.summary[binding.SUMMARY_FIELDS.index("n_episodes")].item()) > 0


def test_gae_noalloc_without_summary_and_limits():
    T, N = 5, 600
    a, b = _pair(T, N, 13)
    d = synth.make_world(2, n_envs=N)
    ctx = binding.Context(d, max_envs=N, critic=False)
    ctx.gae(a, 0.97, 0.9, summary=False)
    ctx.close()
    binding.gae_noalloc(b, 0.97, 0.9, summary=False)
    torch.cuda.synchronize()
    for k in OUT:
        assert torch.equal(getattr(a, k), getattr(b, k)), k
    s = b.struct(synth.GAMMA, synth.LAMBDA)
    s.n_envs = binding.IM_GAE_NOALLOC_MAX_ENVS + 1
    s.ld = s.n_envs
    with pytest.raises(binding.ImError, match="IM_GAE_NOALLOC_MAX_ENVS") as ei:
        binding.im_gae_noalloc(s)
    assert ei.value.status == binding.IM_ERR_UNSUPPORTED
    s = b.struct(synth.GAMMA, synth.LAMBDA)
    s.T = 0
    with pytest.raises(binding.ImError, match="T must"):
        binding.im_gae_noalloc(s)
