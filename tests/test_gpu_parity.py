"""GPU parity of the HIP path (through the C ABI) against the CPU oracle, at
sizes the oracle finishes in seconds: every element compared.

Covered: RNG words (bit-exact) and Gaussians (1e-6 * max|z|) from the
inspection call; PerturbParameters and its +eps/-2eps/+eps triple
(Algorithm 1); the fused K-seed apply loop with records in the kernel
arguments and staged in device memory; the late-joiner replay (Appendix B);
ragged, tiny and mixed-dtype tensors; the identity cases; independence of the
result from how tensors are grouped.
"""
import numpy as np
import pytest

import oracle
from paper_2306_10015_amd import synth
from gpu_util import assert_theta_close, to_device, to_host, z_close

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


SEEDS = [(0, 0, 0), (1, 0, 0), (2**40 + 7, 3, 9), (2**64 - 1, 2**32 - 1, 2**32 - 1)]


@pytest.mark.parametrize("seed", SEEDS)
def test_rng_words_bit_exact(mz, orc, seed):
    for tid in (0, 5, 2**32 - 1):
        for first, count in [(0, 4096), (3, 1001), (2**34 - 1000, 1000), (123456789, 77), (7, 1)]:
            w, _ = mz.debug_generate(seed, tid, first, count, z=False)
            sync()
            ref, _ = orc.generate(seed, tid, first, count, z=False)
            got = w.cpu().numpy().view(np.uint32)
            assert np.array_equal(got, ref), (seed, tid, first, count)


def test_gaussians_within_tolerance(mz, orc):
    n = 1 << 22
    worst = 0.0
    for seed, tid, first in [((0, 0, 0), 0, 0), ((77, 5, 3), 9, 2**33 + 2)]:
        _, z = mz.debug_generate(seed, tid, first, n, words=False)
        sync()
        _, ref = orc.generate(seed, tid, first, n, words=False)
        got = z.cpu().numpy()
        s = z_close(got, ref)
        print(f"z parity seed={seed}: max abs err {s['max_abs_err']:.3e} (tol {s['tol']:.3e})")
        worst = max(worst, s["max_abs_err"] / s["tol"])
        assert s["max_abs_err"] <= s["tol"]
    print(f"worst z error / tolerance = {worst:.3f}")


def make_set(mz, hosts, ids=None):
    devs = [to_device(h) for h in hosts]
    return devs, mz.ParamSet(devs, ids)


def tiny_hosts(dtype):
    w = synth.WORKLOADS["tiny"]
    return [synth.theta0_tensor(s, dtype, i, 0) for i, (_, s) in enumerate(w.shapes)]


def step_and_check(devs, tids, gpu_op, oracle_op, what):
    """Run one GPU operation and check it against the oracle applied to the
    same input (the GPU's own state before the step)."""
    before = [to_host(d) for d in devs]
    gpu_op()
    sync()
    out = None
    for i, (d, b) in enumerate(zip(devs, before)):
        ref = oracle_op(b.copy(), tids[i])
        out = assert_theta_close(to_host(d), ref, f"{what} tensor {i}", inp=b)
    return out


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
def test_perturb_triple_tiny(mz, orc, dtype):
    hosts = tiny_hosts(dtype)
    devs, ps = make_set(mz, hosts)
    seed, eps = (0, 0, 0), 1e-3
    for c in (eps, -2 * eps, eps):
        s = step_and_check(devs, range(len(devs)), lambda: ps.perturb(seed, c),
                           lambda th, tid: orc.perturb(th, tid, seed, c), f"perturb {c:+g}")
        print(f"{dtype} perturb {c:+g}: {s}")
    # the whole triple against the oracle's own triple
    ref = [h.copy() for h in hosts]
    for c in (eps, -2 * eps, eps):
        for i, r in enumerate(ref):
            orc.perturb(r, i, seed, c)
    got = np.concatenate([to_host(d) for d in devs])
    want = np.concatenate(ref)
    exact = float(np.mean(got == want))
    print(f"{dtype} triple: fraction equal to the oracle's triple bit for bit = {exact:.6f}")
    if dtype == synth.BF16:
        # correct RNE on store: nearly every element matches bit for bit
        assert exact > 0.999


def test_perturb_of_zero_is_z(mz, orc):
    n = 10007
    devs, ps = make_set(mz, [np.zeros(n, dtype=np.float32)], [3])
    ps.perturb((5, 1, 2), 1.0)
    sync()
    _, z = orc.generate((5, 1, 2), 3, 0, n)
    s = z_close(to_host(devs[0]), z)
    assert s["max_abs_err"] <= s["tol"]


@pytest.mark.parametrize("dtype,K", [(synth.F32, 4), (synth.BF16, 4), (synth.F32, 40),
                                     (synth.BF16, 64)])
def test_update_multi_tiny(mz, orc, dtype, K):
    hosts = tiny_hosts(dtype)
    devs, ps = make_set(mz, hosts)
    seeds = synth.seeds(K, 1)
    q = synth.grads_int8(K, "uniform", seed=1)
    lr = 1e-3 if dtype == synth.BF16 else 1e-6
    ps.update_multi(seeds, q, lr)
    sync()
    for i, (d, h) in enumerate(zip(devs, hosts)):
        ref = orc.update(h.copy(), i, seeds, q, lr)
        s = assert_theta_close(to_host(d), ref, f"update K={K} tensor {i}", inp=h)
    print(f"{dtype} update K={K}: {s}")


@pytest.mark.parametrize("alpha", [oracle.LOG2_ALPHA, 1.0])
def test_update_signed_log_codec(mz, orc, alpha):
    """The signed-log code with a base-2 log (default) and the natural log."""
    hosts = tiny_hosts(synth.F32)[:1]
    devs, ps = make_set(mz, hosts)
    seeds = synth.seeds(4, 2, step=11)
    q = synth.grads_int8(8, "normal40", seed=4) // 8
    cd = mz.codec(mz.SIGNED_LOG, 1.0, alpha)
    ps.update_multi(seeds, q, 1e-4, cd)
    sync()
    ref = orc.update(hosts[0].copy(), 0, seeds, q, 1e-4, oracle.SIGNED_LOG, 1.0, alpha)
    assert_theta_close(to_host(devs[0]), ref, "signed-log update")


def ragged_hosts():
    sizes = [1, 2, 3, 5, 7, 8, 9, 15, 17, 4095, 4097, 2048 * 3 + 5, 4096 * 2 + 3, 70001]
    hosts = []
    for i, n in enumerate(sizes):
        dt = synth.F32 if i % 2 == 0 else synth.BF16
        hosts.append(synth.theta0_tensor((n,), dt, i, 5))
    ids = [1000 - 7 * i for i in range(len(sizes))]
    return hosts, ids


def test_ragged_mixed_dtype_update_and_perturb(mz, orc):
    hosts, ids = ragged_hosts()
    devs, ps = make_set(mz, hosts, ids)
    seeds = synth.seeds(3, 3, step=2)
    q = synth.grads_int8(9, seed=8)
    step_and_check(devs, ids, lambda: ps.perturb((9, 9, 9), 1e-3),
                   lambda th, tid: orc.perturb(th, tid, (9, 9, 9), 1e-3), "ragged perturb")
    step_and_check(devs, ids, lambda: ps.update_multi(seeds, q, 1e-3),
                   lambda th, tid: orc.update(th, tid, seeds, q, 1e-3), "ragged update")


def test_flat_buffer_views(mz, orc):
    """Tensors as 16-byte-aligned views of one flat allocation."""
    import torch
    sizes = [1000, 4, 777, 4096, 13]
    offs, o = [], 0
    for n in sizes:
        offs.append(o)
        o += (n + 3) // 4 * 4
    flat_h = synth.theta0_tensor((o,), synth.F32, 0, 9)
    flat = to_device(flat_h)
    views = [flat[a:a + n] for a, n in zip(offs, sizes)]
    ps = mz.ParamSet(views)
    seeds = synth.seeds(2, 2)
    q = synth.grads_int8(4, seed=2)
    ps.update_multi(seeds, q, 1e-2)
    torch.cuda.synchronize()
    got = to_host(flat)
    for i, (a, n) in enumerate(zip(offs, sizes)):
        ref = orc.update(flat_h[a:a + n].copy(), i, seeds, q, 1e-2)
        assert_theta_close(got[a:a + n], ref, f"view {i}")
    # padding between views is untouched
    for a, n in zip(offs, sizes):
        pad = slice(a + n, a + (n + 3) // 4 * 4)
        assert np.array_equal(got[pad], flat_h[pad])


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
def test_replay_matches_oracle_and_sequential_updates(mz, orc, dtype):
    ids = [0, 1, 2]
    hosts = [synth.theta0_tensor((n,), dtype, i, 3) for i, n in enumerate([5000, 4097, 33])]
    T = 6
    steps = [(synth.seeds(2, 3, step=t), synth.grads_int8(6, seed=50 + t), 1e-3 * (t + 1))
             for t in range(T)]
    devs, ps = make_set(mz, hosts, ids)
    ps.replay(steps)
    devs2, ps2 = make_set(mz, hosts, ids)
    for t, (s, q, lr) in enumerate(steps):
        step_and_check(devs2, ids, lambda: ps2.update_multi(s, q, lr),
                       lambda th, tid: orc.update(th, tid, s, q, lr), f"replay step {t}")
    for i, (h, d, d2) in enumerate(zip(hosts, devs, devs2)):
        a, b = to_host(d), to_host(d2)
        assert np.array_equal(a.view(np.uint8), b.view(np.uint8)), "replay != sequential updates"
        ref = orc.replay(h.copy(), ids[i], steps)
        if dtype == synth.F32:
            assert_theta_close(a, ref, f"replay tensor {i}")
        else:
            from gpu_util import bf16_ulp_distance
            hist = np.bincount(bf16_ulp_distance(a, ref))
            print(f"bf16 replay vs oracle replay, ulp histogram: {hist[:4]}")


def test_replay_long_log_staged(mz, orc):
    """More records than fit in the kernel arguments (staged buffer), reused
    across six calls on the same paramset: bit-identical to the same steps
    applied one update_multi call at a time (records in the kernel arguments),
    each of which is checked against the oracle on its own input."""
    hosts = [synth.theta0_tensor((3001,), synth.BF16, 0, 4)]
    devs, ps = make_set(mz, hosts)
    devs_seq, ps_seq = make_set(mz, hosts)
    for call in range(6):
        steps = [(synth.seeds(4, 4, step=100 * call + t), synth.grads_int8(16, seed=call * 10 + t),
                  5e-3) for t in range(5)]
        ps.replay(steps)
        for t, (s, q, lr) in enumerate(steps):
            step_and_check(devs_seq, [0], lambda: ps_seq.update_multi(s, q, lr),
                           lambda th, tid: orc.update(th, tid, s, q, lr), f"call {call} step {t}")
    sync()
    assert np.array_equal(to_host(devs[0]), to_host(devs_seq[0]))


def test_replay_split_into_launches_at_step_ends(mz, orc):
    """A log of more records than one launch takes (65536) runs as several
    launches split at step ends, and a single step longer than that runs as a
    launch of its own: the result is bit-identical to the same steps applied
    one update_multi call at a time, and sampled elements after the long step
    match the oracle."""
    n = 1 << 16
    hosts = [synth.theta0_tensor((n,), synth.F32, 0, 8)]
    steps = [(synth.seeds(32, 32, step=t), synth.grads_int8(1024, seed=300 + t), 1e-5)
             for t in range(66)]                       # 67584 records in all
    devs, ps = make_set(mz, hosts)
    ps.replay(steps)
    devs_seq, ps_seq = make_set(mz, hosts)
    for s, q, lr in steps:
        ps_seq.update_multi(s, q, lr)
    sync()
    assert np.array_equal(to_host(devs[0]).view(np.uint32), to_host(devs_seq[0]).view(np.uint32))
    long_step = (synth.seeds(70, 1000, step=900), synth.grads_int8(70000, seed=901), 1e-6)
    tail = [(synth.seeds(4, 4, step=902 + t), synth.grads_int8(16, seed=903 + t), 1e-4) for t in range(3)]
    idx = np.random.Generator(np.random.PCG64(5)).choice(n, 96, replace=False).astype(np.uint64)
    before = to_host(devs[0])[idx.astype(np.int64)]
    ps.replay([tail[0], long_step] + tail[1:])
    for s, q, lr in [tail[0], long_step] + tail[1:]:
        ps_seq.update_multi(s, q, lr)
    sync()
    got = to_host(devs[0])
    assert np.array_equal(got.view(np.uint32), to_host(devs_seq[0]).view(np.uint32))
    ref = orc.replay(before.copy(), 0, [tail[0], long_step] + tail[1:], idx=idx)
    assert_theta_close(got[idx.astype(np.int64)], ref, "replay with a 70000-record step", inp=before)


@pytest.mark.parametrize("case", ["lr0", "q0", "K0", "scale0"])
def test_identity_cases_bit_exact(mz, case):
    hosts = tiny_hosts(synth.F32)[:2]
    hosts[0][::5] = -0.0
    devs, ps = make_set(mz, hosts)
    seeds = synth.seeds(4, 1)
    q = synth.grads_int8(4, seed=3)
    if case == "lr0":
        ps.update_multi(seeds, q, 0.0)
    elif case == "q0":
        ps.update_multi(seeds, np.zeros(4, dtype=np.int8), 1.0)
    elif case == "K0":
        ps.update_multi(seeds[:0], q[:0], 1.0)
    else:
        ps.perturb((1, 2, 3), 0.0)
    sync()
    for h, d in zip(hosts, devs):
        assert np.array_equal(to_host(d).view(np.uint32), h.view(np.uint32))


def test_zero_codes_are_dropped(mz, orc):
    hosts = tiny_hosts(synth.F32)[:1]
    devs, ps = make_set(mz, hosts)
    seeds = synth.seeds(6, 1)
    q = np.array([0, 5, 0, -7, 0, 0], dtype=np.int8)
    ps.update_multi(seeds, q, 1e-2)
    sync()
    ref = orc.update(hosts[0].copy(), 0, seeds, q, 1e-2)
    assert_theta_close(to_host(devs[0]), ref, "zero codes")


def test_grouping_does_not_change_any_bit(mz):
    hosts, ids = ragged_hosts()
    seeds = synth.seeds(4, 2)
    q = synth.grads_int8(8, seed=12)
    devs_all, ps_all = make_set(mz, hosts, ids)
    ps_all.update_multi(seeds, q, 1e-2)
    rev = list(reversed(range(len(hosts))))
    devs_rev, ps_rev = make_set(mz, [hosts[i] for i in rev], [ids[i] for i in rev])
    ps_rev.update_multi(seeds, q, 1e-2)
    singles = []
    for h, tid in zip(hosts, ids):
        d, p = make_set(mz, [h], [tid])
        p.update_multi(seeds, q, 1e-2)
        singles.append(d[0])
    sync()
    for j, i in enumerate(rev):
        a = to_host(devs_all[i]).view(np.uint8)
        assert np.array_equal(a, to_host(devs_rev[j]).view(np.uint8))
        assert np.array_equal(a, to_host(singles[i]).view(np.uint8))


def test_streams_are_respected(mz, orc):
    import torch
    hosts = tiny_hosts(synth.F32)[:1]
    devs, ps = make_set(mz, hosts)
    s = torch.cuda.Stream()
    torch.cuda.current_stream().synchronize()
    with torch.cuda.stream(s):
        ps.perturb((1, 1, 1), 1e-3)
        ps.update_multi(synth.seeds(40, 1), synth.grads_int8(40, seed=6), 1e-4)
    s.synchronize()
    ref = orc.perturb(hosts[0].copy(), 0, (1, 1, 1), 1e-3)
    orc.update(ref, 0, synth.seeds(40, 1), synth.grads_int8(40, seed=6), 1e-4)
    assert_theta_close(to_host(devs[0]), ref, "side stream")


# ---- out of place: the backup restore fused into the sweep ----------------

def test_update_from_backup_matches_oracle_and_leaves_source(mz, orc):
    hosts, ids = ragged_hosts()
    backup_devs, backup = make_set(mz, hosts, ids)
    zeros = [np.zeros_like(h) for h in hosts]
    devs, ps = make_set(mz, zeros, ids)
    seeds = synth.seeds(4, 2, step=3)
    q = synth.grads_int8(8, seed=21)
    ps.update_multi_from(backup, seeds, q, 2e-3)
    sync()
    for h, d, b, tid in zip(hosts, devs, backup_devs, ids):
        ref = orc.update(h.copy(), tid, seeds, q, 2e-3)
        assert_theta_close(to_host(d), ref, f"update_from n={h.size}", inp=h)
        assert np.array_equal(to_host(b).view(np.uint8), h.view(np.uint8))


def test_perturb_from_and_zero_weight_copy(mz, orc):
    hosts, ids = ragged_hosts()
    hosts[0][0] = -0.0
    backup_devs, backup = make_set(mz, hosts, ids)
    devs, ps = make_set(mz, [np.ones_like(h) for h in hosts], ids)
    ps.perturb_from(backup, (7, 1, 2), 1e-3)
    sync()
    for h, d, tid in zip(hosts, devs, ids):
        ref = orc.perturb(h.copy(), tid, (7, 1, 2), 1e-3)
        assert_theta_close(to_host(d), ref, f"perturb_from n={h.size}", inp=h)
    ps.update_multi_from(backup, synth.seeds(2, 1), np.zeros(2, dtype=np.int8), 1.0)
    sync()
    for h, d in zip(hosts, devs):
        assert np.array_equal(to_host(d).view(np.uint8), h.view(np.uint8))


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
def test_algorithm1_iteration_restore_fused(mz, orc, dtype):
    """Backup, perturb triple in place (drifts), then the fused restore+update
    gives exactly what copying the backup back and updating in place gives."""
    import torch
    hosts = [synth.theta0_tensor((n,), dtype, i, 8) for i, n in enumerate([70001, 4096, 33])]
    devs, ps = make_set(mz, hosts)
    backup_devs, backup = make_set(mz, hosts)
    s, eps = (0, 5, 0), 1e-3
    for c in (eps, -2 * eps, eps):
        ps.perturb(s, c)
    seeds = synth.seeds(8, 1, step=5)
    q = synth.grads_int8(8, seed=31)
    ps.update_multi_from(backup, seeds, q, 1e-3)
    ref_devs, ref_ps = make_set(mz, hosts)
    ref_ps.update_multi(seeds, q, 1e-3)
    torch.cuda.synchronize()
    for i, (d, r, h) in enumerate(zip(devs, ref_devs, hosts)):
        assert np.array_equal(to_host(d).view(np.uint8), to_host(r).view(np.uint8))
        assert_theta_close(to_host(d), orc.update(h.copy(), i, seeds, q, 1e-3), f"tensor {i}", inp=h)


def float_class(a):
    """Per element: 1 = +inf, -1 = -inf, 2 = NaN, 0 = finite (fp32 values or
    bf16 bit patterns)."""
    if a.dtype == np.float32:
        return np.where(np.isnan(a), 2, np.where(np.isposinf(a), 1, np.where(np.isneginf(a), -1, 0)))
    special = ((a >> 7) & 0xFF) == 0xFF
    nan = special & ((a & 0x7F) != 0)
    inf = special & ((a & 0x7F) == 0)
    return np.where(nan, 2, np.where(inf, np.where(a >> 15, -1, 1), 0))


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
def test_non_finite_weights_stay_non_finite(mz, orc, dtype):
    """Weights holding +inf, -inf and NaN (a diverged model): a perturbation
    and an update leave each of them +inf, -inf or NaN as it was, and every
    finite weight within the bar of the oracle applied to the same input."""
    h = synth.theta0_tensor((9001,), dtype, 0, 3)
    special = [0, 17, 4095, 4096, 8999, 9000]
    if dtype == synth.F32:
        h[special] = np.array([np.inf, -np.inf, np.nan, np.inf, -np.nan, -np.inf], np.float32)
    else:
        h[special] = np.array([0x7F80, 0xFF80, 0x7FC0, 0x7F80, 0xFFC1, 0xFF80], np.uint16)
    devs, ps = make_set(mz, [h])
    s = (5, 5, 5)
    seeds, q = synth.seeds(6, 1, step=4), synth.grads_int8(6, seed=9)
    ps.perturb(s, 1e-3)
    ps.update_multi(seeds, q, 1e-3)
    sync()
    got = to_host(devs[0])
    assert np.array_equal(float_class(got), float_class(h))
    finite = float_class(h) == 0
    ref = orc.update(orc.perturb(h.copy(), 0, s, 1e-3), 0, seeds, q, 1e-3)
    mid = orc.perturb(h.copy(), 0, s, 1e-3)
    assert_theta_close(got[finite], ref[finite], f"finite weights ({dtype})", inp=mid[finite])


# ---- checksum (ChecksumMatch, Algorithm 1) ---------------------------------

def test_checksum_matches_oracle_and_is_additive(mz, orc):
    hosts, ids = ragged_hosts()
    devs, ps = make_set(mz, hosts, ids)
    want = orc.checksum(hosts, ids)
    assert ps.checksum() == want
    half = len(hosts) // 2
    _, a = make_set(mz, hosts[:half], ids[:half])
    _, b = make_set(mz, hosts[half:], ids[half:])
    assert (a.checksum() + b.checksum()) & 0xFFFFFFFFFFFFFFFF == want
    # after GPU work the checksum is that of the bits the GPU holds
    ps.update_multi(synth.seeds(3, 1), synth.grads_int8(3, seed=5), 1e-2)
    sync()
    assert ps.checksum() == orc.checksum([to_host(d) for d in devs], ids)


def test_checksum_detects_one_flipped_bit(mz):
    import torch
    hosts = tiny_hosts(synth.BF16)
    devs, ps = make_set(mz, hosts)
    base = ps.checksum()
    raw = devs[2].view(torch.int16)
    raw[123457] ^= 1
    assert ps.checksum() != base
    raw[123457] ^= 1
    assert ps.checksum() == base


def test_checksum_on_a_side_stream(mz, orc):
    """checksum(stream=s) returns the checksum of theta after the work queued
    before it on s (it waits for s, not for the current stream)."""
    import torch
    hosts = tiny_hosts(synth.F32)
    devs, ps = make_set(mz, hosts)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        ps.replay([(synth.seeds(8, 4, step=t), synth.grads_int8(32, seed=t), 1e-4) for t in range(40)])
    got = ps.checksum(stream=s)
    torch.cuda.synchronize()
    assert got == orc.checksum([to_host(d) for d in devs])


def test_checksums_of_one_set_on_many_streams(mz, orc):
    """Checksum calls of one paramset (fp32 and bf16 tensors: two launches a
    call, each of hundreds of workgroups) queued twice on each of 20 streams
    with no ordering between them, more streams than the paramset tracks (so
    entries change stream after a host wait): each stream's calls sum in the
    running sum of its own entry, every result equals the oracle's, and the
    sums are left at zero (later calls on the current stream agree)."""
    import torch
    f32, bf16 = tiny_hosts(synth.F32), tiny_hosts(synth.BF16)
    hosts = [f32[0], bf16[1], f32[2], bf16[3]]
    devs, ps = make_set(mz, hosts)
    want = orc.checksum(hosts)
    assert ps.checksum() == want
    streams = [torch.cuda.Stream() for _ in range(20)]
    outs = torch.zeros((20, 2), dtype=torch.int64, device="cuda")
    torch.cuda.synchronize()
    for rep in range(2):
        for k, s in enumerate(streams):
            ps.checksum_into(outs[k, rep:rep + 1], stream=s)
    torch.cuda.synchronize()
    got = [int(v) & 0xFFFFFFFFFFFFFFFF for v in outs.flatten().tolist()]
    assert got == [want] * 40
    assert ps.checksum() == want and ps.checksum() == want


def test_checksum_full_125m_set(mz, orc):
    import torch
    from gpu_util import theta_on_device
    w = synth.WORKLOADS["opt125m"]
    tensors = theta_on_device(w, seed=3, device_rng=True)
    ps = mz.ParamSet(tensors)
    got = ps.checksum()
    assert got == orc.checksum([to_host(t) for t in tensors])
    ps.close()
    del tensors
    torch.cuda.empty_cache()


# ---- element-range shards ---------------------------------------------------

SHARD_CUTS = [0, 24000, 50016, 70001]   # multiples of 8; the last shard ragged


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
def test_shards_compute_the_whole_tensors(mz, orc, dtype):
    """Two tensors split by element range into three shards each, shard k of
    both in paramset k (what one GPU of a sharded run holds). A perturb, a
    staged 40-seed update and a replay give on the shards, bit for bit, the
    whole tensors' result; the shards' checksums add up to the whole set's;
    and a shard's perturb matches the oracle at its elements' global
    indices."""
    n = SHARD_CUTS[-1]
    hosts = [synth.theta0_tensor((n,), dtype, 5 + i, 0) for i in range(2)]
    ids = [11, 4]
    whole_devs, whole = make_set(mz, hosts, ids)
    shard_devs, shards = [], []
    for k in range(3):
        a, b = SHARD_CUTS[k], SHARD_CUTS[k + 1]
        devs = [to_device(h[a:b].copy()) for h in hosts]
        shard_devs.append(devs)
        shards.append(mz.ParamSet(devs, ids, firsts=[a, a]))
    # one perturb: the middle shard against the oracle at global indices
    for ps in [whole] + shards:
        ps.perturb((3, 1, 0), 1e-3)
    sync()
    a, b = SHARD_CUTS[1], SHARD_CUTS[2]
    for i, tid in enumerate(ids):
        ref = orc.perturb(hosts[i][a:b].copy(), tid, (3, 1, 0), 1e-3, first=a)
        assert_theta_close(to_host(shard_devs[1][i]), ref, f"shard at {a}", inp=hosts[i][a:b])
    seeds = synth.seeds(8, 5, step=2)
    q = synth.grads_int8(40, seed=8)
    log = [(synth.seeds(4, 2, step=t), synth.grads_int8(8, seed=30 + t), 1e-3) for t in range(3)]
    for ps in [whole] + shards:
        ps.update_multi(seeds, q, 1e-3)
        ps.replay(log)
    sync()
    for i in range(len(hosts)):
        got = np.concatenate([to_host(shard_devs[k][i]) for k in range(3)])
        assert np.array_equal(got.view(np.uint8), to_host(whole_devs[i]).view(np.uint8))
    assert sum(ps.checksum() for ps in shards) & 0xFFFFFFFFFFFFFFFF == whole.checksum()


def test_shard_offset_is_part_of_the_backup_layout(mz):
    """The out-of-place calls need the same offsets in source and destination."""
    h = synth.theta0_tensor((64,), synth.F32, 0, 0)
    _, a = make_set(mz, [h])
    b = mz.ParamSet([to_device(h)], [0], firsts=[8])
    with pytest.raises(mz.MezoError) as e:
        b.perturb_from(a, (1, 1, 1), 1e-3)
    assert e.value.code == mz.EINVAL


# ---- HIP graph capture ------------------------------------------------------

@pytest.mark.filterwarnings("ignore:The CUDA Graph is empty")  # the refused capture records nothing
def test_graph_capture_of_inline_calls(mz):
    """A perturb, a 4-seed update and a checksum captured into a HIP graph
    (after the paramset's first call): each of three replays, with eager work
    and synchronisations in between, applies them again, bit-identical to the
    same calls made eagerly on a twin set. During capture a staged record
    list is refused before anything is enqueued."""
    import torch
    hosts = [tiny_hosts(synth.F32)[0], tiny_hosts(synth.BF16)[1]]
    devs, ps = make_set(mz, hosts)
    twin_devs, twin = make_set(mz, hosts)
    seeds, q = synth.seeds(4, 1, step=7), synth.grads_int8(4, seed=3)
    for p in (ps, twin):
        p.perturb((9, 9, 9), 1e-3)   # the first call creates the device tables
    ck = torch.zeros(1, dtype=torch.int64, device="cuda")
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        ps.perturb((1, 2, 3), 1e-3)
        ps.update_multi(seeds, q, 1e-3)
        ps.checksum_into(ck)
    torch.cuda.synchronize()
    for _ in range(3):
        g.replay()
        twin.perturb((1, 2, 3), 1e-3)
        twin.update_multi(seeds, q, 1e-3)
        torch.cuda.synchronize()
        torch.randn(4096, device="cuda").sum().item()   # eager work between replays
        for d, t in zip(devs, twin_devs):
            assert torch.equal(d.view(torch.int16), t.view(torch.int16))
        assert int(ck.item()) & 0xFFFFFFFFFFFFFFFF == twin.checksum()
    g2 = torch.cuda.CUDAGraph()
    with pytest.raises(mz.MezoError) as e:
        with torch.cuda.graph(g2):
            ps.update_multi(synth.seeds(8, 5), synth.grads_int8(40, seed=1), 1e-3)
    assert e.value.code == mz.EINVAL
    torch.cuda.synchronize()


# ---- log edge cases and concurrent callers ---------------------------------

@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
def test_replay_with_empty_and_zero_steps(mz, orc, dtype):
    """A log holding an all-zero step, an empty step, a zero-lr step and a step
    with some zero codes: bit-identical to the same steps as update_multi
    calls (dropped steps do nothing, not even a rounding) and, in fp32, to the
    oracle's replay within the bar."""
    hosts = [synth.theta0_tensor((n,), dtype, i, 8) for i, n in enumerate([4097, 70])]
    s = [synth.seeds(3, 1, step=t) for t in range(6)]
    steps = [(s[0], synth.grads_int8(3, seed=1), 1e-3),
             (s[1], np.zeros(3, np.int8), 1e-3),
             (s[2][:0], np.zeros(0, np.int8), 1e-3),
             (s[3], synth.grads_int8(3, seed=4), 0.0),
             (s[4], np.array([0, 9, 0], np.int8), 2e-3),
             (s[5], synth.grads_int8(3, seed=6), 1e-3)]
    devs, ps = make_set(mz, hosts)
    ps.replay(steps)
    devs2, ps2 = make_set(mz, hosts)
    for seeds, q, lr in steps:
        ps2.update_multi(seeds, q, lr)
    sync()
    for i, (h, a, b) in enumerate(zip(hosts, devs, devs2)):
        ga = to_host(a)
        assert np.array_equal(ga.view(np.uint8), to_host(b).view(np.uint8))
        if dtype == synth.F32:
            assert_theta_close(ga, orc.replay(h.copy(), i, steps), f"replay with empty steps, tensor {i}")


def test_concurrent_callers_on_separate_paramsets(mz):
    """Four host threads, each driving its own paramset on its own stream
    (perturbs, inline and staged updates, replays, checksums), give the same
    bits as the same work done by one thread."""
    import threading
    import torch

    def work(ps, stream, k, out):
        with torch.cuda.stream(stream):
            for it in range(5):
                ps.perturb((k, it, 0), 1e-3)
                ps.update_multi(synth.seeds(40, 1, step=it), synth.grads_int8(40, seed=k * 10 + it), 1e-4)
                ps.replay([(synth.seeds(8, 1, step=100 + it + j), synth.grads_int8(8, seed=j), 1e-4)
                           for j in range(6)])
                ps.perturb((k, it, 0), -1e-3)
            out[k] = ps.checksum(stream)

    def run(parallel):
        sets, streams, out = [], [], {}
        for k in range(4):
            hosts = [synth.theta0_tensor((n,), dt, i, k) for i, (n, dt) in
                     enumerate([(20000, synth.F32), (9001, synth.BF16)])]
            sets.append(make_set(mz, hosts))
            streams.append(torch.cuda.Stream())
        torch.cuda.synchronize()
        if parallel:
            threads = [threading.Thread(target=work, args=(sets[k][1], streams[k], k, out)) for k in range(4)]
            for t in threads:
                t.start()
            for t in threads:
                t.join()
        else:
            for k in range(4):
                work(sets[k][1], streams[k], k, out)
        torch.cuda.synchronize()
        return out, [[to_host(d) for d in devs] for devs, _ in sets]

    seq_sums, seq_vals = run(False)
    par_sums, par_vals = run(True)
    assert seq_sums == par_sums
    for a, b in zip(seq_vals, par_vals):
        for x, y in zip(a, b):
            assert np.array_equal(x.view(np.uint8), y.view(np.uint8))


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
@pytest.mark.parametrize("n", [2, 37])
def test_perturb_multi_is_sequential_perturbs(mz, orc, dtype, n):
    """n perturbs in one pass (inline and staged records) are bit-identical
    to n perturb calls, and match the oracle's sequential perturbs."""
    hosts = [synth.theta0_tensor((m,), dtype, i, 9) for i, m in enumerate([5003, 2048, 17])]
    rng = np.random.Generator(np.random.PCG64(n))
    seeds = [(int(rng.integers(0, 4)), int(rng.integers(0, 100)), int(rng.integers(0, 16))) for _ in range(n)]
    scales = (rng.choice([1e-3, -2e-3, 0.0, 5e-4], size=n)).astype(np.float32)
    devs, ps = make_set(mz, hosts)
    ps.perturb_multi(seeds, scales)
    devs2, ps2 = make_set(mz, hosts)
    for sd, sc in zip(seeds, scales):
        ps2.perturb(sd, float(sc))
    sync()
    for i, (h, a, b) in enumerate(zip(hosts, devs, devs2)):
        ga = to_host(a)
        assert np.array_equal(ga.view(np.uint8), to_host(b).view(np.uint8))
        if dtype == synth.F32:
            ref = h.copy()
            for sd, sc in zip(seeds, scales):
                orc.perturb(ref, i, sd, float(sc))
            assert_theta_close(ga, ref, f"perturb_multi tensor {i}")


def test_perturb_multi_nf4_portable_bit_exact(mz, orc):
    """Restore sample j and perturb for sample j + 1 in one pass on 4-bit
    storage: bit-identical to the oracle's two perturbs (portable mode)."""
    import torch
    from oracle import nf4
    n = 4097
    p, a = synth.nf4_theta0_tensor(n, 0)
    t = mz.NF4Tensor(torch.from_numpy(p.copy()).cuda(), torch.from_numpy(a.copy()).cuda(), n)
    ps = mz.ParamSet([t], [4], gaussian=mz.GAUSS_PORTABLE)
    seeds, scales = [(1, 5, 3), (1, 5, 4)], [1e-3, 1e-3]
    ps.perturb_multi(seeds, scales)
    sync()
    c, am = nf4.unpack(p, n), a
    for sd, sc in zip(seeds, scales):
        c, am = nf4.perturb(c, am, 4, sd, sc, portable=True)
    assert np.array_equal(t.codes.cpu().numpy(), nf4.pack(c))
    assert np.array_equal(t.absmax.cpu().numpy().view(np.uint32), am.view(np.uint32))
    ps.close()


def test_more_streams_than_tracked(mz, orc):
    """One paramset driven from 20 streams in a chain (each waits for the one
    before): more streams than the paramset tracks, so later streams take over
    the entries used longest ago. The result is the chain's, bit for bit (the
    portable Gaussian), and destroy returns with every stream drained."""
    import torch
    hosts = tiny_hosts(synth.F32)[:1]
    devs, ps = make_set(mz, hosts)
    ps.set_gaussian(mz.GAUSS_PORTABLE)
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream() for _ in range(20)]
    prev = torch.cuda.current_stream()
    ref = hosts[0].copy()
    for i, s in enumerate(streams):
        s.wait_stream(prev)
        with torch.cuda.stream(s):
            ps.perturb((i, 1, 0), 1e-3)
        orc.perturb(ref, 0, (i, 1, 0), 1e-3, portable=True)
        prev = s
    ps.close()
    assert all(s.query() for s in streams)
    assert np.array_equal(to_host(devs[0]).view(np.uint32), ref.view(np.uint32))


def test_destroy_waits_for_work_on_every_stream(mz):
    """A paramset used on two streams: destroy returns only after the long
    replay on the first stream has finished, not just the short perturb
    enqueued last on the second."""
    import torch
    w = synth.WORKLOADS["opt125m"]
    hosts = [synth.theta0_tensor((1 << 24,), synth.F32, 0, 1)]
    devs, ps = make_set(mz, hosts)
    a, b = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    log = [(synth.seeds(8, 4, step=t), synth.grads_int8(32, seed=t), 1e-6) for t in range(40)]
    with torch.cuda.stream(a):
        ps.replay(log)                      # 1280 records: tens of milliseconds
    with torch.cuda.stream(b):
        ps.perturb((1, 2, 3), w.eps)        # short, enqueued last
    ps.close()
    assert a.query() and b.query()
    torch.cuda.synchronize()
