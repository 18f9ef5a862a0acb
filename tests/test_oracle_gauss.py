"""Pins of the oracle's Gaussian draw z ~ N(0,1) (Algorithm 1,
PerturbParameters): closed-form special cases of the Box-Muller transform on
hand-picked words, the transform's defining identities, and statistical bounds
(mean 0, variance 1, normal shape) over millions of draws."""
import math

import numpy as np
import pytest

R_MAX = math.sqrt(48.0 * math.log(2.0))  # u1 = 2^-24: sqrt(-2 ln 2^-24)


def words(a_top24, b_top24, c_top24, d_top24, low=0):
    """Words whose top 24 bits are given (low 8 bits = `low`)."""
    return np.array([(v << 8) | low for v in (a_top24, b_top24, c_top24, d_top24)],
                    dtype=np.uint32)


def test_u1_one_gives_zero_radius(orc):
    z = orc.box_muller(words(2**24 - 1, 12345, 2**24 - 1, 777))
    assert np.all(z == 0.0)


def test_u1_smallest_gives_max_radius_and_u2_zero_gives_cos_branch(orc):
    z = orc.box_muller(words(0, 0, 0, 0))
    assert z[0] == pytest.approx(R_MAX, rel=1e-15) and z[1] == 0.0
    assert z[2] == pytest.approx(R_MAX, rel=1e-15) and z[3] == 0.0


def test_low_byte_is_ignored(orc):
    a = orc.box_muller(words(5, 6, 7, 8, low=0))
    b = orc.box_muller(words(5, 6, 7, 8, low=0xFF))
    assert np.array_equal(a, b)


@pytest.mark.parametrize("quarter, cos_sign, sin_sign", [(1, 0, 1), (2, -1, 0), (3, 0, -1)])
def test_phase_quarters(orc, quarter, cos_sign, sin_sign):
    """u2 = k/4 puts the point on an axis: (cos, sin) = (0,1), (-1,0), (0,-1)."""
    z = orc.box_muller(words(0, quarter << 22, 2**24 - 1, 0))
    assert z[0] == pytest.approx(cos_sign * R_MAX, abs=1e-14)
    assert z[1] == pytest.approx(sin_sign * R_MAX, abs=1e-14)
    assert z[2] == 0.0 and z[3] == 0.0  # second pair has u1 = 1: radius 0


def test_pairs_use_their_own_words(orc):
    """(w0, w1) drive z0, z1 and (w2, w3) drive z2, z3: changing w2/w3 leaves
    z0/z1 alone and vice versa."""
    base = orc.box_muller(words(100, 200, 300, 400))
    c = orc.box_muller(words(100, 200, 301, 999))
    d = orc.box_muller(words(555, 666, 300, 400))
    assert np.array_equal(base[:2], c[:2]) and not np.array_equal(base[2:], c[2:])
    assert np.array_equal(base[2:], d[2:]) and not np.array_equal(base[:2], d[:2])


def test_radius_and_angle_identities(orc):
    """z0^2 + z1^2 = -2 ln u1 and atan2(z1, z0) = 2 pi u2 (mod 2 pi)."""
    rng = np.random.Generator(np.random.PCG64(5))
    for _ in range(1000):
        w = rng.integers(0, 2**32, size=4, dtype=np.uint64).astype(np.uint32)
        z = orc.box_muller(w)
        for p in range(2):
            u1 = ((int(w[2 * p]) >> 8) + 1) / 2**24
            u2 = (int(w[2 * p + 1]) >> 8) / 2**24
            r2 = z[2 * p] ** 2 + z[2 * p + 1] ** 2
            assert r2 == pytest.approx(-2.0 * math.log(u1), rel=1e-12, abs=1e-15)
            if r2 > 1e-12:
                ang = math.atan2(z[2 * p + 1], z[2 * p]) % (2 * math.pi)
                d = abs(ang - 2 * math.pi * u2)
                assert min(d, 2 * math.pi - d) < 1e-9


def test_element_z_is_fp32_of_its_block_slot(orc):
    seed = (3, 1, 2)
    _, z = orc.generate(seed, 2, 40, 16)
    for i in range(16):
        e = 40 + i
        zz = orc.box_muller(orc.block_words(seed, 2, e))
        assert z[i] == np.float32(zz[e & 3])


@pytest.fixture(scope="module")
def big_sample(orc):
    n = 1 << 22
    _, z = orc.generate((0, 0, 0), 0, 0, n, words=False, z=True)
    return z.astype(np.float64)


def test_mean_and_variance(big_sample):
    z = big_sample
    n = z.size
    assert abs(z.mean()) <= 5 / math.sqrt(n)
    assert abs(z.var() - 1.0) <= 5 * math.sqrt(2.0 / n)


def test_normal_shape_ks_and_kurtosis(big_sample):
    from scipy import stats
    z = big_sample
    n = z.size
    d = stats.kstest(z, "norm").statistic
    assert d <= 1.63 / math.sqrt(n), d
    assert abs(stats.kurtosis(z, fisher=False) - 3.0) < 0.02
    assert np.abs(z).max() <= R_MAX * (1 + 1e-6)


def test_no_correlation_between_seeds_and_within_pairs(orc, big_sample):
    n = big_sample.size
    _, z2 = orc.generate((1, 0, 0), 0, 0, n, words=False, z=True)
    bound = 5 / math.sqrt(n)
    assert abs(np.corrcoef(big_sample, z2.astype(np.float64))[0, 1]) <= bound
    pairs = big_sample.reshape(-1, 2)
    assert abs(np.corrcoef(pairs[:, 0], pairs[:, 1])[0, 1]) <= 5 / math.sqrt(n // 2)
    quads = big_sample.reshape(-1, 4)
    assert abs(np.corrcoef(quads[:, 0], quads[:, 2])[0, 1]) <= 5 / math.sqrt(n // 4)


def test_block_array_forms_equal_the_single_block_forms(orc):
    """The oracle's many-block Box-Muller (fast and portable) is its
    single-block transform applied block by block (fp64 rounded once to fp32
    for the fast one)."""
    rng = np.random.Generator(np.random.PCG64(77))
    w = rng.integers(0, 2**32, size=4 * 500, dtype=np.uint64).astype(np.uint32)
    w[:8] = [0, 0, 0xFFFFFFFF, 0xFFFFFFFF, 0xFF, 0x100, 0x80000000, 0x7FFFFF00]
    z = orc.box_muller_blocks(w)
    zp = orc.box_muller_blocks(w, portable=True)
    for b in range(500):
        blk = w[4 * b:4 * b + 4]
        assert np.array_equal(z[4 * b:4 * b + 4], orc.box_muller(blk).astype(np.float32))
        assert np.array_equal(zp[4 * b:4 * b + 4], orc.box_muller_portable(blk))
