"""GPU parity at the size limit: one tensor of MEZO_MAX_NUMEL = 2^34 elements
(the Philox counter's block index e >> 2 reaches 2^32 - 1), in bf16 (32 GiB)
and in 4-bit storage (8 GiB of codes, 1 GiB of absmax). The tensor is zeroed,
seeded windows (its first and last elements and random blocks in between)
get seeded values, and those windows are compared with the oracle after a
perturb and an update."""
import numpy as np
import pytest

from paper_2306_10015_amd import synth
from gpu_util import assert_theta_close, to_host

pytestmark = pytest.mark.gpu

N = 1 << 34


@pytest.fixture(scope="module")
def mz():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    from paper_2306_10015_amd import mezo
    return mezo


def windows(rng, n_blocks, block, count):
    """Start indices (multiples of `block`) of the first, last and random blocks."""
    mid = rng.integers(1, n_blocks - 1, size=count)
    return np.unique(np.concatenate([[0, n_blocks - 1], mid])) * block


def test_max_size_bf16(mz, orc):
    import torch
    assert mz.MAX_NUMEL == N
    t = torch.zeros(N, dtype=torch.bfloat16, device="cuda")
    rng = np.random.Generator(np.random.PCG64(21))
    starts = windows(rng, N // 4096, 4096, 14)
    idx = (starts[:, None] + np.arange(4096)[None, :]).ravel().astype(np.int64)
    vals = synth.theta0_tensor((idx.size,), synth.BF16, 3)
    ix_dev = torch.from_numpy(idx).cuda()
    t.index_copy_(0, ix_dev, torch.from_numpy(vals.view(np.int16)).view(torch.bfloat16).cuda())
    ps = mz.ParamSet([t], [77])
    s = (5, 9, 2)
    ps.perturb(s, 1e-3)
    torch.cuda.synchronize()
    got = to_host(t.index_select(0, ix_dev))
    want = orc.perturb(vals.copy(), 77, s, 1e-3, idx=idx.astype(np.uint64))
    assert_theta_close(got, want, "perturb at 2^34", inp=vals)
    before = got
    seeds = synth.seeds(4, 1, step=1)
    q = synth.grads_int8(4, seed=2)
    ps.update_multi(seeds, q, 1e-3)
    torch.cuda.synchronize()
    got = to_host(t.index_select(0, ix_dev))
    want = orc.update(before.copy(), 77, seeds, q, 1e-3, idx=idx.astype(np.uint64))
    assert_theta_close(got, want, "update at 2^34", inp=before)
    ps.close()
    del t
    torch.cuda.empty_cache()


def test_max_size_nf4(mz, orc):
    import torch
    from oracle import nf4
    codes = torch.zeros(N // 2, dtype=torch.uint8, device="cuda")
    absmax = torch.zeros(N // 64, dtype=torch.float32, device="cuda")
    rng = np.random.Generator(np.random.PCG64(22))
    blocks = windows(rng, N // 64, 1, 30)
    byte_ix = (blocks[:, None] * 32 + np.arange(32)[None, :]).ravel().astype(np.int64)
    packed, am = synth.nf4_theta0_tensor(blocks.size * 64, 5)
    bdev = torch.from_numpy(byte_ix).cuda()
    adev = torch.from_numpy(blocks.astype(np.int64)).cuda()
    codes.index_copy_(0, bdev, torch.from_numpy(packed).cuda())
    absmax.index_copy_(0, adev, torch.from_numpy(am).cuda())
    ps = mz.ParamSet([mz.NF4Tensor(codes, absmax, N)], [3], gaussian=mz.GAUSS_PORTABLE)
    seeds = synth.seeds(4, 1, step=2)
    q = synth.grads_int8(4, seed=3)
    ps.update_multi(seeds, q, 5e-3)
    torch.cuda.synchronize()
    got_c = nf4.unpack(codes.index_select(0, bdev).cpu().numpy(), blocks.size * 64)
    got_a = absmax.index_select(0, adev).cpu().numpy()
    c_ref, a_ref = nf4.update(nf4.unpack(packed, blocks.size * 64), am, 3, seeds, q, 5e-3,
                              numel=N, blocks=blocks, portable=True)
    assert np.array_equal(got_a.view(np.uint32), a_ref.view(np.uint32))
    assert np.array_equal(got_c, c_ref)
    ps.close()
    del codes, absmax
    torch.cuda.empty_cache()
