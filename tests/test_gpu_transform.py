"""The Gaussian transform checked over every value of each uniform. Box-Muller
is separable: the radius depends on u1 alone, the angle on u2 alone, and z is
their product, so two sweeps reach every radius and every angle: all 2^24
values of u1 (at two fixed angles) and all 2^24 values of u2 (at two fixed
radii). The GPU's fast transform stays within 1e-6 * max|z| of the oracle's
fp64 value on both sweeps, which bounds its error for every pair of words;
the portable transform is bit-exact on both. The low bytes of the words,
which the definition ignores, are filled with noise."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

N = 1 << 24


@pytest.fixture(scope="module")
def mz():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    from paper_2306_10015_amd import mezo
    return mezo


def sweep_words(kind):
    rng = np.random.Generator(np.random.PCG64(1 if kind == "u1" else 2))
    t = np.arange(N, dtype=np.uint32) << 8
    w = np.zeros(4 * N, dtype=np.uint32)
    if kind == "u1":
        # pair 0: every u1 at angle 0; pair 1: every u1 at a quarter turn
        w[0::4], w[1::4] = t, 0
        w[2::4], w[3::4] = t, (1 << 22) << 8
    else:
        # pair 0: every u2 at the largest radius (u1 = 2^-24); pair 1: u1 = 1/2
        w[0::4], w[1::4] = 0, t
        w[2::4], w[3::4] = ((1 << 23) - 1) << 8, t
    return w | rng.integers(0, 256, size=w.size, dtype=np.uint64).astype(np.uint32)


def gpu_z(mz, words, gaussian):
    import torch
    dev = torch.from_numpy(words.view(np.int32)).cuda()
    z = mz.debug_box_muller(dev, gaussian)
    torch.cuda.synchronize()
    return z.cpu().numpy()


@pytest.mark.parametrize("kind", ["u1", "u2"])
def test_fast_transform_over_every_input(mz, orc, kind):
    w = sweep_words(kind)
    got = gpu_z(mz, w, mz.GAUSS_FAST).astype(np.float64)
    ref = orc.box_muller_blocks(w).astype(np.float64)
    err = np.abs(got - ref)
    tol = 1e-6 * np.max(np.abs(ref))
    big = np.abs(ref) > 0.01
    ulps = err[big] / np.spacing(np.abs(ref[big]).astype(np.float32)).astype(np.float64)
    print(f"fast transform, every {kind}: max abs err {err.max():.3e} (tol {tol:.3e}), "
          f"bit-exact {np.mean(err == 0):.4f}, where |z| > 0.01: 99.9th percentile "
          f"{np.percentile(ulps, 99.9):.1f} ulp, max {ulps.max():.1f} ulp")
    assert err.max() <= tol


@pytest.mark.parametrize("kind", ["u1", "u2"])
def test_portable_transform_is_bit_exact_over_every_input(mz, orc, kind):
    w = sweep_words(kind)
    got = gpu_z(mz, w, mz.GAUSS_PORTABLE)
    ref = orc.box_muller_blocks(w, portable=True)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))
