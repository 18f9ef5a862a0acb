"""Pins of the oracle's portable Gaussian (binary32 operations only; Appendix
B's requirement that every device regenerate the same noise) and of the
binary32 update that goes with it: closeness to the textbook fp64
Box-Muller value, the octant special cases, the normal shape, and the update's
relations to perturb, replay and the reference update."""
import math

import numpy as np
import pytest

from paper_2306_10015_amd import synth

R_MAX = math.sqrt(48.0 * math.log(2.0))


def words(a_top24, b_top24, c_top24=2**24 - 1, d_top24=0):
    return np.array([(v << 8) for v in (a_top24, b_top24, c_top24, d_top24)], dtype=np.uint32)


def test_close_to_the_fp64_box_muller(orc):
    n = 1 << 21
    for seed in [(0, 0, 0), (123456789, 7, 3)]:
        _, ref = orc.generate(seed, 4, 1000, n, words=False)
        _, por = orc.generate(seed, 4, 1000, n, words=False, portable=True)
        err = np.abs(por.astype(np.float64) - ref.astype(np.float64))
        assert err.max() <= 1e-6 * np.abs(ref).max()
        ulps = np.abs(por.astype(np.float64) - ref) / np.spacing(np.maximum(np.abs(ref), 1e-30))
        assert np.percentile(ulps, 99.99) <= 4


def test_radius_and_axes_special_cases(orc):
    z = orc.box_muller_portable(words(2**24 - 1, 12345))       # u1 = 1: r = 0
    assert z[0] == 0.0 and z[1] == 0.0
    z = orc.box_muller_portable(words(0, 0))                   # u1 = 2^-24, angle 0
    assert z[0] == pytest.approx(R_MAX, rel=2e-7) and z[1] == 0.0
    for quarter, (cs, sn) in {1: (0, 1), 2: (-1, 0), 3: (0, -1)}.items():
        z = orc.box_muller_portable(words(0, quarter << 22))
        assert z[0] == pytest.approx(cs * R_MAX, abs=1e-6)
        assert z[1] == pytest.approx(sn * R_MAX, abs=1e-6)
    # octant boundaries: the angle is continuous across every eighth of a turn
    for k in range(1, 8):
        lo = orc.box_muller_portable(words(1000, (k << 21) - 1))
        hi = orc.box_muller_portable(words(1000, k << 21))
        assert abs(lo[0] - hi[0]) < 1e-5 and abs(lo[1] - hi[1]) < 1e-5


def test_radius_identity_and_angle(orc):
    rng = np.random.Generator(np.random.PCG64(51))
    for _ in range(2000):
        w = rng.integers(0, 2**32, size=4, dtype=np.uint64).astype(np.uint32)
        z = orc.box_muller_portable(w).astype(np.float64)
        u1 = ((int(w[0]) >> 8) + 1) / 2**24
        u2 = (int(w[1]) >> 8) / 2**24
        assert z[0] ** 2 + z[1] ** 2 == pytest.approx(-2 * math.log(u1), rel=2e-6, abs=1e-12)
        if -2 * math.log(u1) > 1e-6:
            ang = math.atan2(z[1], z[0]) % (2 * math.pi)
            d = abs(ang - 2 * math.pi * u2)
            assert min(d, 2 * math.pi - d) < 1e-5


def test_normal_shape(orc):
    from scipy import stats
    n = 1 << 22
    _, z = orc.generate((9, 9, 9), 1, 0, n, words=False, portable=True)
    z = z.astype(np.float64)
    assert abs(z.mean()) <= 5 / math.sqrt(n)
    assert abs(z.var() - 1) <= 5 * math.sqrt(2 / n)
    assert stats.kstest(z, "norm").statistic <= 1.63 / math.sqrt(n)


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
def test_portable_update_relations(orc, dtype):
    n = 20000
    th0 = synth.theta0_tensor((n,), dtype, 3)
    seeds = synth.seeds(4, 2, step=1)
    q = synth.grads_int8(8, seed=4)
    lr = 1e-3
    a = orc.update(th0.copy(), 2, seeds, q, lr, portable=True)
    b = orc.update(th0.copy(), 2, seeds, q, lr)
    if dtype == synth.F32:
        assert np.max(np.abs(a.astype(np.float64) - b)) <= 1e-6 * np.abs(b).max()
    else:
        ordered = [np.where(x.astype(np.int64) & 0x8000, -(x.astype(np.int64) & 0x7FFF),
                            x.astype(np.int64)) for x in (a, b)]
        assert np.mean(np.abs(ordered[0] - ordered[1]) <= 1) > 0.9999
    # one record: the update is the perturb with scale c
    c = orc.coefficients(q[:1], lr)
    p1 = orc.perturb(th0.copy(), 2, seeds[0], float(c[0]), portable=True)
    u1 = orc.update(th0.copy(), 2, seeds[:1], q[:1], lr, portable=True)
    assert np.array_equal(p1, u1)
    # replay = updates in sequence
    steps = [(synth.seeds(2, 2, step=t), synth.grads_int8(4, seed=60 + t), 1e-3) for t in range(4)]
    r = orc.replay(th0.copy(), 2, steps, portable=True)
    s = th0.copy()
    for ss, qq, ll in steps:
        orc.update(s, 2, ss, qq, ll, portable=True)
    assert np.array_equal(r, s)


def test_portable_update_accumulates_in_binary32_order(orc):
    """On a zero tensor with two records the result is fl32(fma(c1, z1,
    fl32(c0 z0))): the documented binary32 order, checked with numpy's
    correctly rounded float32 arithmetic on the oracle's own z."""
    n = 4096
    seeds = synth.seeds(2, 1)
    q = np.array([90, -55], dtype=np.int8)
    lr = 0.5
    got = orc.update(np.zeros(n, np.float32), 0, seeds, q, lr, portable=True)
    c = orc.coefficients(q, lr)
    _, z0 = orc.generate(seeds[0], 0, 0, n, words=False, portable=True)
    _, z1 = orc.generate(seeds[1], 0, 0, n, words=False, portable=True)
    acc0 = (np.float64(c[0]) * z0.astype(np.float64)).astype(np.float32)      # fma(c0, z0, 0)
    acc1 = (np.float64(c[1]) * z1.astype(np.float64) + acc0).astype(np.float32)  # one rounding
    # the fp64 sum of an exact product and a float32 is exact enough that its
    # single rounding equals fma's except in double-rounding corner cases
    assert np.mean(got == acc1) > 0.9999
