"""The GPU measurement probes (include/instantmimic_calib.h): each runs, and
its checksums equal what its documented access pattern gives, computed here on
the CPU -- so the figures the bench derives from them are of the work stated."""
import numpy as np
import pytest
import torch

from paper_2609_09821_amd import binding

pytestmark = pytest.mark.gpu


def _lds_words():
    return (np.arange(65536 // 4, dtype=np.uint64) * 2654435761) & 0xFFFFFFFF


def _lds_expected(width, waves):
    w = _lds_words().astype(np.uint32)
    out = np.zeros(64 * waves, np.uint32)
    for wave in range(waves):
        for lane in range(64):
            x = 0
            for s in range(16):
                if width == 16:
                    r = (wave * 32 + s * 8 + (lane & 31)) & 511
                    q = (2 * (s & 3) + (lane >> 5)) & 7
                    off = r * 128 + ((q ^ ((r >> 1) & 7)) * 16)
                else:
                    off = ((wave * 16 + s) * 512 + lane * 8) & 65535
                for k in range(width // 4):
                    x ^= int(w[off // 4 + k])
            out[wave * 64 + lane] = x
    return out


@pytest.mark.parametrize("width,waves", [(16, 4), (16, 16), (8, 2)])
def test_lds_probe_reads_the_documented_words(width, waves):
    blocks = 3
    out = torch.zeros(64 * waves * blocks, dtype=torch.int32, device="cuda")
    binding.im_calib_lds(width, waves, 1, blocks, out.data_ptr())
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(np.uint32).reshape(blocks, 64 * waves)
    exp = _lds_expected(width, waves)
    for b in range(blocks):
        assert np.array_equal(got[b], exp)
    # an even number of rounds XORs every word twice
    binding.im_calib_lds(width, waves, 2, blocks, out.data_ptr())
    torch.cuda.synchronize()
    assert not out.cpu().numpy().any()


def test_read_probe_reads_every_word_once_per_pass():
    nbytes, blocks = 1 << 20, 2
    T = 256 * blocks
    words = torch.arange(nbytes // 4, dtype=torch.int32, device="cuda")
    out = torch.zeros(T, dtype=torch.int32, device="cuda")
    binding.im_calib_read(words.data_ptr(), nbytes, 1, blocks, out.data_ptr())
    torch.cuda.synchronize()
    w = np.arange(nbytes // 4, dtype=np.uint32).reshape(-1, 4)       # 16-byte words
    per_word = w[:, 0] ^ w[:, 1] ^ w[:, 2] ^ w[:, 3]
    exp = np.zeros(T, np.uint32)
    for t in range(T):
        exp[t] = np.bitwise_xor.reduce(per_word[t::T])
    assert np.array_equal(out.cpu().numpy().view(np.uint32), exp)


@pytest.mark.parametrize("kind", [binding.IM_CALIB_MFMA_BF16, binding.IM_CALIB_MFMA_F32])
def test_mfma_probe_work_is_linear_in_the_rounds(kind):
    # every accumulator grows by the same product each round, so the per-thread
    # checksums of 2 rounds are twice those of 1 (up to fp32 rounding)
    blocks = 4
    o1 = torch.zeros(256 * blocks, device="cuda")
    o2 = torch.zeros(256 * blocks, device="cuda")
    binding.im_calib_mfma(kind, 1, blocks, o1.data_ptr())
    binding.im_calib_mfma(kind, 2, blocks, o2.data_ptr())
    torch.cuda.synchronize()
    a, b = o1.cpu().numpy(), o2.cpu().numpy()
    assert np.isfinite(a).all() and np.abs(a).sum() > 0
    np.testing.assert_allclose(b, 2 * a, rtol=1e-6)
