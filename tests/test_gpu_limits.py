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


def test_generate_across_its_launch_chunks(mz, orc):
    """mezo_debug_generate splits a range into launches of 2^28 elements: a
    range starting mid-block just below 2^28 and longer than one launch gives
    the oracle's words and z at its ends and around the split."""
    import torch
    from gpu_util import Z_REL
    first, count = (1 << 28) - 6, (1 << 28) + 20
    seed = (2 ** 40 + 3, 9, 4)
    w, z = mz.debug_generate(seed, 17, first, count)
    torch.cuda.synchronize()
    # the start, the split (local element 2^28) and the end, inside [0, count)
    for a, n in ((0, 64), ((1 << 28) - 32, 48), (count - 64, 64)):
        assert a + n <= count
        ww, zz = orc.generate(seed, 17, first + a, n)
        assert np.array_equal(w[a:a + n].cpu().numpy().view(np.uint32), ww)
        ref = zz.astype(np.float64)
        err = np.abs(z[a:a + n].cpu().numpy().astype(np.float64) - ref)
        assert err.max() <= Z_REL * max(np.abs(ref).max(), 1.0)
    del w, z
    torch.cuda.empty_cache()


def test_box_muller_across_its_launch_chunks(mz, orc):
    """mezo_debug_box_muller splits its blocks into launches of 2^26: blocks on
    both sides of the split match the oracle (the portable transform bit for
    bit)."""
    import torch
    n_blocks = (1 << 26) + 5
    g = torch.Generator(device="cuda")
    g.manual_seed(5)
    words = torch.randint(-(1 << 31), 1 << 31, (4 * n_blocks,), dtype=torch.int64, device="cuda",
                          generator=g).to(torch.int32)
    z = mz.debug_box_muller(words, mz.GAUSS_PORTABLE)
    torch.cuda.synchronize()
    for b0 in (0, (1 << 26) - 3, n_blocks - 4):
        wb = words[4 * b0:4 * (b0 + 4)].cpu().numpy().view(np.uint32)
        got = z[4 * b0:4 * (b0 + 4)].cpu().numpy()
        assert np.array_equal(got.view(np.uint32), orc.box_muller_blocks(wb, portable=True).view(np.uint32))
    del words, z
    torch.cuda.empty_cache()
