"""The portable mode on the GPU is bit-identical to the CPU oracle's binary32
definition (Appendix B: every device regenerates the same noise): the
Gaussians themselves, and the weights after perturb, fused updates and replay,
for fp32 and bf16 storage, small ragged sets, the full 125M set and the full
6.7B bf16 set (sampled elements) with an update and a replay that move the
weights."""
import numpy as np
import pytest

from paper_2306_10015_amd import synth
from gpu_util import theta_on_device, to_device, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mz():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    from paper_2306_10015_amd import mezo
    return mezo


def sync():
    import torch
    torch.cuda.synchronize()


def bits(a):
    return a.view(np.uint32) if a.dtype == np.float32 else a


@pytest.mark.parametrize("seed,tid,first", [((0, 0, 0), 0, 0), ((2**40 + 3, 9, 4), 77, 2**33 + 1),
                                            ((2**64 - 1, 2**32 - 1, 2**32 - 1), 2**32 - 1, 5)])
def test_portable_gaussians_bit_exact(mz, orc, seed, tid, first):
    n = 1 << 21
    _, z = mz.debug_generate(seed, tid, first, n, words=False, gaussian=mz.GAUSS_PORTABLE)
    sync()
    _, ref = orc.generate(seed, tid, first, n, words=False, portable=True)
    got = z.cpu().numpy()
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))


def portable_set(mz, hosts, ids=None):
    devs = [to_device(h) for h in hosts]
    return devs, mz.ParamSet(devs, ids, gaussian=mz.GAUSS_PORTABLE)


def ragged():
    sizes = [1, 3, 8, 9, 4095, 4097, 70001, 2048 * 3 + 5]
    hosts = [synth.theta0_tensor((n,), synth.F32 if i % 2 == 0 else synth.BF16, i, 6)
             for i, n in enumerate(sizes)]
    return hosts, [500 + 3 * i for i in range(len(sizes))]


def test_portable_perturb_update_replay_bit_exact(mz, orc):
    hosts, ids = ragged()
    devs, ps = portable_set(mz, hosts, ids)
    refs = [h.copy() for h in hosts]
    s, eps = (4, 2, 1), 1e-3
    for c in (eps, -2 * eps, eps):
        ps.perturb(s, c)
        for r, tid in zip(refs, ids):
            orc.perturb(r, tid, s, c, portable=True)
    seeds = synth.seeds(5, 2, step=9)
    q = synth.grads_int8(10, seed=12)
    ps.update_multi(seeds, q, 3e-3)
    for r, tid in zip(refs, ids):
        orc.update(r, tid, seeds, q, 3e-3, portable=True)
    steps = [(synth.seeds(3, 3, step=20 + t), synth.grads_int8(9, seed=70 + t), 1e-3) for t in range(6)]
    ps.replay(steps)                     # 54 records: staged path
    for r, tid in zip(refs, ids):
        orc.replay(r, tid, steps, portable=True)
    sync()
    for h, d, r in zip(hosts, devs, refs):
        assert np.array_equal(bits(to_host(d)), bits(r)), f"n={h.size}"


def test_portable_from_backup_bit_exact(mz, orc):
    hosts, ids = ragged()
    bdevs, backup = portable_set(mz, hosts, ids)
    devs, ps = portable_set(mz, [np.zeros_like(h) for h in hosts], ids)
    seeds = synth.seeds(4, 1)
    q = synth.grads_int8(4, seed=3)
    ps.update_multi_from(backup, seeds, q, 1e-2)
    sync()
    for h, d, tid in zip(hosts, devs, ids):
        ref = orc.update(h.copy(), tid, seeds, q, 1e-2, portable=True)
        assert np.array_equal(bits(to_host(d)), bits(ref))


def test_portable_subnormal_weights_and_scales_bit_exact(mz, orc):
    """Subnormal weights (fp32 and bf16 storage), a perturbation of subnormal
    scale and an update whose coefficients are subnormal: the results, still
    mostly subnormal, equal the oracle's bit for bit (denormals kept on both
    sides; a flush to zero anywhere on the GPU would show)."""
    rng = np.random.Generator(np.random.PCG64(41))
    n = 4097
    sign32 = rng.integers(0, 2, n, dtype=np.uint32) << np.uint32(31)
    f = (rng.integers(1, 1 << 23, n, dtype=np.uint32) | sign32).view(np.float32)
    sign16 = (rng.integers(0, 2, n, dtype=np.uint16) << np.uint16(15)).astype(np.uint16)
    b = (rng.integers(1, 1 << 7, n, dtype=np.uint16) | sign16).astype(np.uint16)
    hosts, ids = [f, b], [3, 8]
    devs, ps = portable_set(mz, hosts, ids)
    refs = [h.copy() for h in hosts]
    s = (6, 1, 0)
    ps.perturb(s, 1e-39)
    for r, tid in zip(refs, ids):
        orc.perturb(r, tid, s, 1e-39, portable=True)
    seeds = synth.seeds(3, 1, step=2)
    q = synth.grads_int8(3, seed=4)
    ps.update_multi(seeds, q, 1e-40)
    for r, tid in zip(refs, ids):
        orc.update(r, tid, seeds, q, 1e-40, portable=True)
    sync()
    for h, d, r in zip(hosts, devs, refs):
        assert np.array_equal(bits(to_host(d)), bits(r)), f"{h.dtype}"
    tiny = np.finfo(np.float32).tiny
    assert np.mean((refs[0] != 0) & (np.abs(refs[0]) < tiny)) > 0.5
    assert not np.array_equal(bits(refs[0]), bits(f)) and not np.array_equal(refs[1], b)


def test_portable_full_125m_update_bit_exact(mz, orc):
    import torch
    w = synth.WORKLOADS["opt125m"]
    tensors = theta_on_device(w, seed=1, device_rng=True)
    ps = mz.ParamSet(tensors, gaussian=mz.GAUSS_PORTABLE)
    rng = np.random.Generator(np.random.PCG64(8))
    idx = [synth.sample_indices(t.numel(), rng, edge=512, blocks=16) for t in tensors]

    def gather():
        return [to_host(t.index_select(0, torch.from_numpy(ix.astype(np.int64)).cuda()))
                for t, ix in zip(tensors, idx)]

    before = gather()
    seeds = synth.workload_seeds(w)
    q = synth.grads_int8(w.K, seed=1)
    ps.perturb((0, 0, 0), w.eps)
    ps.update_multi(seeds, q, w.lr)
    sync()
    after = gather()
    for tid, (b, a, ix) in enumerate(zip(before, after, idx)):
        ref = orc.perturb(b.copy(), tid, (0, 0, 0), w.eps, idx=ix, portable=True)
        orc.update(ref, tid, seeds, q, w.lr, idx=ix, portable=True)
        assert np.array_equal(bits(a), bits(ref)), f"tensor {tid}"
    ps.close()
    del tensors
    torch.cuda.empty_cache()


def test_portable_full_6p7b_update_bit_exact(mz, orc):
    """The 6.7B bf16 set (323 tensors, the bench's launch configuration) in
    portable mode: perturb +eps, then a K = 64 update at lr = 1e-3 (large
    enough that most bf16 weights change), bit-identical to the oracle's
    binary32 definition on every sampled element (the first and last 48 of
    each tensor and 8 random blocks)."""
    import torch
    w = synth.WORKLOADS["opt6.7b"]
    tensors = theta_on_device(w, seed=3, device_rng=True)
    ps = mz.ParamSet(tensors, gaussian=mz.GAUSS_PORTABLE)
    rng = np.random.Generator(np.random.PCG64(9))
    idx = [synth.sample_indices(t.numel(), rng, edge=48, blocks=8) for t in tensors]

    def gather():
        return [to_host(t.index_select(0, torch.from_numpy(ix.astype(np.int64)).cuda()))
                for t, ix in zip(tensors, idx)]

    before = gather()
    seeds = synth.workload_seeds(w)
    q = synth.grads_int8(w.K, seed=4)
    ps.perturb((0, 5, 0), w.eps)
    ps.update_multi(seeds, q, 1e-3)
    sync()
    after = gather()
    changed = total = 0
    for tid, (b, a, ix) in enumerate(zip(before, after, idx)):
        perturbed = orc.perturb(b.copy(), tid, (0, 5, 0), w.eps, idx=ix, portable=True)
        ref = orc.update(perturbed.copy(), tid, seeds, q, 1e-3, idx=ix, portable=True)
        assert np.array_equal(bits(a), bits(ref)), f"tensor {tid}"
        changed += int(np.sum(ref != perturbed))   # moved by the update itself
        total += ref.size
    print(f"opt6.7b portable perturb + K=64 update at lr=1e-3: {total} sampled elements bit-exact, "
          f"{changed} changed by the update")
    assert changed > total // 2
    ps.close()
    del tensors
    torch.cuda.empty_cache()


def test_portable_full_6p7b_replay_bit_exact(mz, orc):
    """The bench's catch-up on the 6.7B bf16 set in portable mode: a replay of
    T = 4 logged steps of K = 64 seeds (256 staged records, rounded to bf16 at
    every step end) at lr = 1e-3, bit-identical to the oracle's step-by-step
    binary32 replay on every sampled element."""
    import torch
    w = synth.WORKLOADS["opt6.7b"]
    tensors = theta_on_device(w, seed=5, device_rng=True)
    ps = mz.ParamSet(tensors, gaussian=mz.GAUSS_PORTABLE)
    rng = np.random.Generator(np.random.PCG64(10))
    idx = [synth.sample_indices(t.numel(), rng, edge=32, blocks=8) for t in tensors]

    def gather():
        return [to_host(t.index_select(0, torch.from_numpy(ix.astype(np.int64)).cuda()))
                for t, ix in zip(tensors, idx)]

    log = [(synth.seeds(w.machines, w.samples_per_machine, step=10_000 + t),
            synth.grads_int8(w.K, "uniform", seed=2000 + t), 1e-3) for t in range(4)]
    before = gather()
    ps.replay(log)
    sync()
    after = gather()
    changed = total = 0
    for tid, (b, a, ix) in enumerate(zip(before, after, idx)):
        ref = orc.replay(b.copy(), tid, log, idx=ix, portable=True)
        assert np.array_equal(bits(a), bits(ref)), f"tensor {tid}"
        changed += int(np.sum(ref != b))
        total += ref.size
    print(f"opt6.7b portable replay 4 x 64: {total} sampled elements bit-exact, {changed} changed")
    assert changed > total // 2
    ps.close()
    del tensors
    torch.cuda.empty_cache()
