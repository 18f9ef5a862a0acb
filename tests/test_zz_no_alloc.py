"""mezo_replay_noalloc, the entry point that allocates nothing, against
mezo_replay, through the C ABI: two calls in a row on the same GPU (the second
with a smaller parameter set and fewer records, so that it runs over the
staging array the first call left behind), each compared bit for bit with
mezo_replay applied to a copy of the same weights; then a call of at most 32
records (kernel arguments only), a call over the limit (refused, weights
untouched) and a set without device tables (refused)."""
import numpy as np
import pytest

from paper_2306_10015_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mz():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    from paper_2306_10015_amd import mezo
    return mezo


def mixed_set(mz, sizes, seed):
    """fp32, bf16 and NF4 tensors of the given sizes (ragged tails), seeded;
    returns (tensors, a function giving a fresh copy of them)."""
    import torch
    from gpu_util import to_device
    out = []
    for i, (n, kind) in enumerate(sizes):
        if kind == "nf4":
            p, a = synth.nf4_theta0_tensor(n, i, seed)
            out.append(mz.NF4Tensor(torch.from_numpy(p.copy()).cuda(), torch.from_numpy(a.copy()).cuda(), n))
        else:
            out.append(to_device(synth.theta0_tensor((n,), kind, i, seed)))
    return out


def clone(mz, tensors):
    return [mz.NF4Tensor(t.codes.clone(), t.absmax.clone(), t.numel()) if isinstance(t, mz.NF4Tensor)
            else t.clone() for t in tensors]


def bits(mz, tensors):
    import torch
    out = []
    for t in tensors:
        if isinstance(t, mz.NF4Tensor):
            out += [t.codes.cpu().numpy(), t.absmax.cpu().numpy().view(np.uint32)]
        elif t.dtype == torch.bfloat16:
            out.append(t.view(torch.int16).cpu().numpy())
        else:
            out.append(t.cpu().numpy().view(np.uint32))
    return out


def log(T, machines, samples, lr, seed):
    return [(synth.seeds(machines, samples, step=100 + t), synth.grads_int8(machines * samples, "uniform",
                                                                            seed=seed + t), lr * (1 + t % 2))
            for t in range(T)]


def check_pair(mz, sizes, seed, steps, gaussian):
    import torch
    a = mixed_set(mz, sizes, seed)
    b = clone(mz, a)
    ps_a = mz.ParamSet(a, gaussian=gaussian)
    ps_b = mz.ParamSet(b, gaussian=gaussian)
    # a paramset's first call creates its device tables (it may allocate)
    ps_a.perturb((9, 0, 0), 1e-3)
    ps_b.perturb((9, 0, 0), 1e-3)
    ps_a.replay_noalloc(steps)
    ps_b.replay(steps)
    torch.cuda.synchronize()
    for x, y in zip(bits(mz, a), bits(mz, b)):
        assert np.array_equal(x, y)
    ps_a.close()
    ps_b.close()


@pytest.mark.parametrize("gaussian", [0, 1])
def test_two_calls_in_a_row_match_replay(mz, gaussian):
    # call 1: 13 tensors, 12 steps x 64 seeds = 768 records through the staging array
    big = [(70001, "f32"), (4096, "bf16"), (1, "f32"), (2049, "bf16"), (64 * 40 + 7, "nf4"), (1023, "f32"),
           (5000, "nf4"), (8, "bf16"), (2048 * 3, "bf16"), (1024 * 5 + 3, "f32"), (63, "nf4"), (9, "bf16"),
           (300000, "bf16")]
    check_pair(mz, big, seed=1, steps=log(12, 16, 4, 1e-3, seed=50), gaussian=gaussian)
    # call 2: a smaller set, 3 steps x 40 seeds = 120 records (the array still
    # holds the first call's 768)
    small = [(3000, "bf16"), (777, "f32"), (130, "nf4")]
    check_pair(mz, small, seed=2, steps=log(3, 10, 4, 1e-3, seed=90), gaussian=gaussian)


def test_short_lists_and_limits(mz):
    import torch
    sizes = [(5000, "f32"), (2500, "bf16")]
    a = mixed_set(mz, sizes, seed=3)
    b = clone(mz, a)
    ps_a, ps_b = mz.ParamSet(a), mz.ParamSet(b)
    # no device tables yet: refused before anything is enqueued
    with pytest.raises(mz.MezoError) as e:
        ps_a.replay_noalloc(log(1, 4, 1, 1e-3, seed=7))
    assert e.value.code == mz.EINVAL
    ps_a.perturb((9, 0, 0), 1e-3)
    ps_b.perturb((9, 0, 0), 1e-3)
    # at most 32 records travel in the engine's arguments
    steps = log(2, 4, 4, 1e-3, seed=11)
    ps_a.replay_noalloc(steps)
    ps_b.replay(steps)
    # over the limit: refused, the weights untouched
    over = [(synth.seeds(65537, 1, step=0), np.ones(65537, dtype=np.int8), 1e-3)]
    with pytest.raises(mz.MezoError) as e:
        ps_a.replay_noalloc(over)
    assert e.value.code == mz.ERANGE
    # exactly the limit: 65536 records in one step
    full = [(synth.seeds(65536, 1, step=1), synth.grads_int8(65536, "uniform", seed=5), 1e-5)]
    ps_a.replay_noalloc(full)
    ps_b.replay(full)
    torch.cuda.synchronize()
    for x, y in zip(bits(mz, a), bits(mz, b)):
        assert np.array_equal(x, y)
    ps_a.close()
    ps_b.close()


@pytest.mark.filterwarnings("ignore:The CUDA Graph is empty")
def test_graph_capture_of_a_long_replay(mz):
    """A replay of 256 records (past what the kernel arguments carry) captured
    into a HIP graph through mezo_replay_noalloc: the staging launches and the
    engine launch are recorded, nothing is allocated, and each of three
    replays, with eager work and synchronisations in between (one of them an
    eager no-alloc call over the same staging array), applies the log again,
    bit-identical to mezo_replay on a twin set."""
    import torch
    sizes = [(70001, "f32"), (4099, "bf16"), (64 * 9 + 5, "nf4")]
    a = mixed_set(mz, sizes, seed=4)
    b = clone(mz, a)
    ps_a, ps_b = mz.ParamSet(a), mz.ParamSet(b)
    ps_a.perturb((9, 0, 0), 1e-3)   # the first call creates the device tables
    ps_b.perturb((9, 0, 0), 1e-3)
    steps = log(4, 16, 4, 1e-3, seed=21)   # 4 x 64 = 256 records
    other = mz.ParamSet(mixed_set(mz, [(3000, "bf16")], seed=5))
    other.perturb((9, 0, 0), 1e-3)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        ps_a.replay_noalloc(steps)
    torch.cuda.synchronize()
    for i in range(3):
        g.replay()
        ps_b.replay(steps)
        torch.cuda.synchronize()
        torch.randn(4096, device="cuda").sum().item()   # eager work between replays
        other.replay_noalloc(log(2, 8, 4, 1e-3, seed=60 + i))   # rewrites the staging array
        torch.cuda.synchronize()
        for x, y in zip(bits(mz, a), bits(mz, b)):
            assert np.array_equal(x, y), f"graph replay {i}"
    for p in (ps_a, ps_b, other):
        p.close()
