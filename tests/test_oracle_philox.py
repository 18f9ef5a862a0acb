"""Pins of the oracle's counter RNG (Philox4x32-10) against things other than
itself: PyTorch's independent header-only Philox engine (a library routine,
compiled here into a test-only program), the published generator's
bijectivity, and determinism (the paper requires the same seed to regenerate
the same perturbation on every machine: Algorithm 1, PerturbParameters;
Appendix B)."""
import os
import subprocess

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def torch_philox(tmp_path_factory):
    torch = pytest.importorskip("torch")
    inc = os.path.join(os.path.dirname(torch.__file__), "include")
    hdr = os.path.join(inc, "ATen", "core", "PhiloxRNGEngine.h")
    if not os.path.exists(hdr):
        pytest.skip("torch's Philox header is not installed")
    exe = str(tmp_path_factory.mktemp("cmp") / "philox_torch_cmp")
    subprocess.run(["g++", "-std=c++17", "-O1", "-I" + inc,
                    os.path.join(HERE, "philox_torch_cmp.cpp"), "-o", exe], check=True)

    def run(triples):
        inp = "".join(f"{s} {q} {o}\n" for s, q, o in triples)
        out = subprocess.run([exe], input=inp, capture_output=True, text=True, check=True)
        return np.array([[int(v) for v in line.split()] for line in out.stdout.splitlines()],
                        dtype=np.uint64).astype(np.uint32)

    return run


def _cases():
    rng = np.random.Generator(np.random.PCG64(11))
    cases = [(0, 0, 0, 0, 0), (1, 0, 0, 0, 0), (0, 1, 0, 0, 0), (0, 0, 1, 0, 0),
             (0, 0, 0, 1, 0), (0, 0, 0, 0, 4), (2**64 - 1, 2**32 - 1, 2**32 - 1, 2**32 - 1, 2**34 - 1),
             (0x123456789ABCDEF0, 7, 3, 5, 1000), (2**32, 0, 0, 0, 0), (2**32 - 1, 0, 0, 0, 0)]
    for _ in range(200):
        cases.append((int(rng.integers(0, 2**63)) * 2 + int(rng.integers(0, 2)),
                      int(rng.integers(0, 2**32)), int(rng.integers(0, 2**32)),
                      int(rng.integers(0, 2**32)), int(rng.integers(0, 2**34))))
    return cases


def test_words_match_torch_philox_engine(orc, torch_philox):
    """Seed (machine, step, sample), tensor t, element e maps to the engine's
    (seed=machine, subsequence=sample | step<<32, offset=(e>>2) | t<<32)."""
    cases = _cases()
    ref = torch_philox([(m, j | (s << 32), (e >> 2) | (t << 32)) for m, s, j, t, e in cases])
    for (m, s, j, t, e), want in zip(cases, ref):
        got = orc.block_words((m, s, j), t, e)
        assert np.array_equal(got, want), (m, s, j, t, e)


def test_raw_block_function_matches_torch(orc, torch_philox):
    rng = np.random.Generator(np.random.PCG64(12))
    ctrs = rng.integers(0, 2**32, size=(64, 4), dtype=np.uint64)
    keys = rng.integers(0, 2**32, size=(64, 2), dtype=np.uint64)
    trip = [(int(k[0]) | (int(k[1]) << 32), int(c[2]) | (int(c[3]) << 32),
             int(c[0]) | (int(c[1]) << 32)) for c, k in zip(ctrs, keys)]
    ref = torch_philox(trip)
    for c, k, want in zip(ctrs, keys, ref):
        assert np.array_equal(orc.philox(c, k), want)


def test_bijection_on_consecutive_counters(orc):
    """Philox is a bijection of the counter for a fixed key: 2^20 consecutive
    blocks give 2^20 distinct 128-bit outputs."""
    n_blocks = 1 << 20
    w, _ = orc.generate((5, 2, 1), 3, 0, 4 * n_blocks, words=True, z=False)
    blocks = w.reshape(-1, 4).astype(np.uint64)
    key = (blocks[:, 0] << np.uint64(32)) | blocks[:, 1]
    key2 = (blocks[:, 2] << np.uint64(32)) | blocks[:, 3]
    packed = np.stack([key, key2], axis=1)
    assert np.unique(packed, axis=0).shape[0] == n_blocks


def test_word_of_element_is_word_e_mod_4_of_its_block(orc):
    seed = (9, 4, 2)
    w, _ = orc.generate(seed, 6, 1000, 64, words=True, z=False)
    for i in range(64):
        e = 1000 + i
        assert w[i] == orc.block_words(seed, 6, e)[e & 3]


def test_determinism_and_seed_sensitivity(orc):
    a, za = orc.generate((1, 2, 3), 0, 0, 4096)
    b, zb = orc.generate((1, 2, 3), 0, 0, 4096)
    assert np.array_equal(a, b) and np.array_equal(za.view(np.uint32), zb.view(np.uint32))
    for other in [((2, 2, 3), 0), ((1, 3, 3), 0), ((1, 2, 4), 0), ((1, 2, 3), 1)]:
        c, _ = orc.generate(other[0], other[1], 0, 4096, z=False)
        assert np.mean(a == c) < 0.01


def test_uniform_top_bytes_chi_square(orc):
    """The top 8 bits of the words are uniform over 256 cells (chi-square, 255
    degrees of freedom, p > 1e-4)."""
    from scipy import stats
    w, _ = orc.generate((3, 0, 0), 0, 0, 1 << 20, words=True, z=False)
    counts = np.bincount((w >> 24).astype(np.int64), minlength=256)
    chi2, p = stats.chisquare(counts)
    assert p > 1e-4, (chi2, p)
