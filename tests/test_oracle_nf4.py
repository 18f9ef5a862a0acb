"""Pins of the oracle's 4-bit (NF4) storage (Section 3's 4-bit forward-only
variant; the format of QLoRA, which the paper cites): the code values against
their published four-decimal table and against the normal quantiles they are
defined by (computed here with math.erf, not with the oracle's scipy), the
quantizer against a brute-force nearest-value search, the storage round trip
and error bound, the nibble order, and the relations of perturb, update and
replay on NF4 storage to the exact perturbation and to each other."""
import math
import os
from pathlib import Path

import numpy as np
import pytest

from paper_2306_10015_amd import synth

GOLDEN = Path(__file__).parent / "golden" / "nf4_values_qlora.txt"


@pytest.fixture(scope="module")
def nf4(orc):
    from oracle import nf4 as m
    return m


def phi(x):
    return 0.5 * (1.0 + math.erf(x / math.sqrt(2.0)))


def phi_inv(p):
    lo, hi = -10.0, 10.0
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if phi(mid) < p:
            lo = mid
        else:
            hi = mid
    return 0.5 * (lo + hi)


def test_values_match_the_published_table(nf4):
    pub = np.loadtxt(GOLDEN, comments="#")
    v = nf4.table().astype(np.float64)
    assert v.shape == (16,) and np.max(np.abs(v - pub)) <= 5.1e-5


def test_values_structure(nf4):
    v = nf4.table()
    assert v.dtype == np.float32
    assert np.all(np.diff(v) > 0)
    assert v[0] == -1.0 and v[15] == 1.0 and v[nf4.ZERO_CODE] == 0.0
    assert np.sum(v < 0) == 7 and np.sum(v > 0) == 8


def test_values_are_normal_quantiles(nf4):
    """Positive value i (of 8) is Phi^-1(p_i) / Phi^-1(delta) with p spaced
    evenly from delta to 1/2; negative value j (of 7) likewise with 8 points."""
    v = nf4.table().astype(np.float64)
    delta = 1.0 - 0.5 * (1.0 / 32.0 + 1.0 / 30.0)
    top = phi_inv(delta)
    p_pos = [delta + (0.5 - delta) * k / 8 for k in range(8)]        # v[15], v[14], ..., v[8]
    p_neg = [delta + (0.5 - delta) * k / 7 for k in range(7)]        # -v[0], ..., -v[6]
    for k, p in enumerate(p_pos):
        assert phi(v[15 - k] * top) == pytest.approx(p, abs=2e-7)
    for k, p in enumerate(p_neg):
        assert phi(-v[k] * top) == pytest.approx(p, abs=2e-7)


def test_midpoints(nf4):
    v = nf4.table()
    m = nf4.midpoints()
    assert m.dtype == np.float32 and m.shape == (15,)
    assert np.all(v[:-1] < m) and np.all(m < v[1:])
    exact = (v[:-1].astype(np.float64) + v[1:].astype(np.float64)) / 2
    assert np.all(np.abs(m.astype(np.float64) - exact) <= np.abs(np.spacing(m)) / 2)


def blocks_of(kind, rng, n):
    if kind == "normal":
        return (rng.standard_normal(n) * 0.02).astype(np.float32)
    if kind == "uniform":
        return rng.uniform(-3, 3, n).astype(np.float32)
    if kind == "heavy":
        return (rng.standard_cauchy(n) * 1e-3).astype(np.float32)
    if kind == "zeros":
        w = (rng.standard_normal(n) * 0.02).astype(np.float32)
        w[rng.random(n) < 0.5] = 0.0
        return w
    raise ValueError(kind)


@pytest.mark.parametrize("kind", ["normal", "uniform", "heavy", "zeros"])
@pytest.mark.parametrize("n", [1, 5, 64, 100, 64 * 37 + 13])
def test_quantize_is_the_nearest_value(nf4, kind, n):
    rng = np.random.Generator(np.random.PCG64(n * 7 + len(kind)))
    w = blocks_of(kind, rng, n)
    codes, absmax = nf4.quantize(w)
    v = nf4.table().astype(np.float64)
    nb = (n + 63) // 64
    assert absmax.shape == (nb,) and codes.shape == (n,)
    for b in range(nb):
        blk = w[64 * b:64 * (b + 1)]
        c = codes[64 * b:64 * (b + 1)]
        a = np.float32(np.max(np.abs(blk)))
        assert absmax[b] == a
        if a == 0:
            assert np.all(c == nf4.ZERO_CODE)
            continue
        x = (blk * (np.float32(1) / a)).astype(np.float64)   # the fp32 x the definition fixes
        d = np.abs(x[:, None] - v[None, :])
        best = np.argmin(d, axis=1)
        srt = np.sort(d, axis=1)
        assert np.all(srt[:, 1] > srt[:, 0])                  # no ties in these draws
        assert np.array_equal(c, best)
        imax = np.argmax(np.abs(blk))
        assert c[imax] in (0, 15)


def test_zero_and_single_value_blocks(nf4):
    c, a = nf4.quantize(np.zeros(70, np.float32))
    assert np.all(c == nf4.ZERO_CODE) and np.all(a == 0)
    w = np.zeros(64, np.float32)
    w[10] = -3.5
    c, a = nf4.quantize(w)
    assert a[0] == np.float32(3.5) and c[10] == 0 and np.all(np.delete(c, 10) == nf4.ZERO_CODE)


def test_round_trip_on_canonical_blocks(nf4):
    """A block with a +-1 code and absmax a dequantizes to values whose
    largest magnitude is a, and quantizes back to the same codes and a."""
    rng = np.random.Generator(np.random.PCG64(3))
    nb = 300
    codes = rng.integers(0, 16, size=nb * 64, dtype=np.uint8)
    codes[::64] = rng.choice([0, 15], size=nb)
    absmax = rng.uniform(1e-4, 10, nb).astype(np.float32)
    w = nf4.dequantize(codes, absmax)
    c2, a2 = nf4.quantize(w)
    assert np.array_equal(c2, codes) and np.array_equal(a2, absmax)


def test_error_bound(nf4):
    rng = np.random.Generator(np.random.PCG64(4))
    w = (rng.standard_normal(64 * 500) * 0.02).astype(np.float32)
    c, a = nf4.quantize(w)
    back = nf4.dequantize(c, a).astype(np.float64)
    half_gap = np.max(np.diff(nf4.table().astype(np.float64))) / 2
    bound = np.repeat(a.astype(np.float64), 64) * half_gap * (1 + 1e-6)
    assert np.all(np.abs(back - w) <= bound)


def test_nibble_order(nf4):
    assert list(nf4.pack(np.array([1, 2, 3], np.uint8))) == [0x21, 0x03]
    rng = np.random.Generator(np.random.PCG64(5))
    for n in (1, 2, 7, 64, 129):
        c = rng.integers(0, 16, size=n, dtype=np.uint8)
        p = nf4.pack(c)
        assert p.size == (n + 1) // 2
        assert np.array_equal(nf4.unpack(p, n), c)


def make(nf4, n, seed=0):
    w = synth.theta0_tensor((n,), "f32", seed)
    return nf4.quantize(w)


def test_identities(nf4):
    c, a = make(nf4, 1000)
    s = synth.seeds(4, 1)
    assert all(np.array_equal(x, y) for x, y in zip(nf4.perturb(c, a, 0, s[0], 0.0), (c, a)))
    q0 = np.zeros(4, np.int8)
    assert all(np.array_equal(x, y) for x, y in zip(nf4.update(c, a, 0, s, q0, 1e-3), (c, a)))
    assert all(np.array_equal(x, y) for x, y in zip(nf4.replay(c, a, 0, []), (c, a)))


@pytest.mark.parametrize("portable", [False, True])
def test_update_is_the_exact_perturbation_quantized(orc, nf4, portable):
    """deq(update) is within half an NF4 gap (of the new absmax) of
    deq(start) + sum c_k z_k, with z from the generator, in fp64."""
    n = 64 * 40 + 9
    c, a = make(nf4, n, 1)
    seeds = synth.seeds(3, 2, step=2)
    q = synth.grads_int8(6, seed=9)
    lr = 2e-3
    c2, a2 = nf4.update(c, a, 5, seeds, q, lr, portable=portable)
    coef = orc.coefficients(q, lr).astype(np.float64)
    exact = nf4.dequantize(c, a).astype(np.float64)
    for s, ck in zip(seeds, coef):
        _, z = orc.generate(tuple(s), 5, 0, n, words=False)
        exact += ck * z.astype(np.float64)
    half_gap = np.max(np.diff(nf4.table().astype(np.float64))) / 2
    lens = nf4.block_lengths(n, np.arange(a2.size))
    bound = np.repeat(a2.astype(np.float64), lens) * half_gap * (1 + 1e-5) + 1e-9
    assert np.all(np.abs(nf4.dequantize(c2, a2) - exact) <= bound)
    assert not np.array_equal(c2, c)


def test_one_record_update_is_the_perturb(orc, nf4):
    c, a = make(nf4, 3000, 2)
    s = synth.seeds(1, 1, step=4)
    q = np.array([77], np.int8)
    lr = 5e-3
    coef = float(orc.coefficients(q, lr)[0])
    u = nf4.update(c, a, 1, s, q, lr)
    p = nf4.perturb(c, a, 1, tuple(s[0]), coef)
    assert np.array_equal(u[0], p[0]) and np.array_equal(u[1], p[1])


def test_replay_quantizes_after_every_step(orc, nf4):
    n = 64 * 20
    c, a = make(nf4, n, 3)
    steps = [(synth.seeds(2, 2, step=t), synth.grads_int8(4, seed=30 + t), 4e-3) for t in range(5)]
    r = nf4.replay(c, a, 2, steps)
    s = (c, a)
    for seeds, q, lr in steps:
        s = nf4.update(s[0], s[1], 2, seeds, q, lr)
    assert np.array_equal(r[0], s[0]) and np.array_equal(r[1], s[1])
    # one fused update over all the records (a single quantization) differs
    all_seeds = np.concatenate([synth.seeds(2, 2, step=t) for t in range(5)])
    all_q = np.concatenate([q for _, q, _ in steps])
    f = nf4.update(c, a, 2, all_seeds, all_q, 4e-3)
    assert not np.array_equal(f[0], r[0])


def test_blocks_are_independent(nf4):
    n = 64 * 30 + 17
    c, a = make(nf4, n, 4)
    s = synth.seeds(2, 1)
    q = synth.grads_int8(2, seed=1)
    full = nf4.update(c, a, 3, s, q, 0.05)
    blocks = np.array([0, 7, 29, 30])
    ix = nf4.block_elements(n, blocks)
    part = nf4.update(c[ix], a[blocks], 3, s, q, 0.05, numel=n, blocks=blocks)
    assert np.array_equal(part[0], full[0][ix]) and np.array_equal(part[1], full[1][blocks])


def test_checksum_image(orc, nf4):
    c, a = make(nf4, 75, 5)
    p = nf4.pack(c)
    img = nf4.image(p, a)
    assert img.size == 40 + 8            # 38 code bytes padded to 40, then 2 absmax values
    base = nf4.checksum_tensor(p, a, 9)
    for byte in range(p.size):
        for bit in (0, 4):
            q = p.copy()
            q[byte] ^= 1 << bit
            assert nf4.checksum_tensor(q, a, 9) != base
    b = a.copy()
    b.view(np.uint32)[1] ^= 1
    assert nf4.checksum_tensor(p, b, 9) != base
    assert nf4.checksum_tensor(p, a, 8) != base


def test_kernel_bin_table_is_the_nearest_value_rule(nf4, tmp_path):
    """The kernels' NF4 quantizer looks codes up in a bin table of
    csrc/nf4.hpp: the floor table (long record lists) or the round-to-nearest
    table, its bin read off one fma (the fast path of short lists and of the
    standalone quantization) or clamped (their general path). Replayed on the host over every float x
    with |x| <= 1 + 2^-22 and over infinities, NaN and out-of-range values,
    each code equals the number of the oracle's midpoints strictly below x."""
    import shutil
    import subprocess
    if shutil.which("g++") is None:
        pytest.skip("needs g++")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    exe = tmp_path / "nf4_table_check"
    subprocess.run(["g++", "-std=c++17", "-O2", "-ffp-contract=off", "-march=x86-64-v3",
                    "-I" + os.path.join(root, "paper_2306_10015_amd", "csrc"),
                    os.path.join(root, "tests", "nf4_table_check.cpp"), "-o", str(exe)], check=True)
    mids = " ".join(f"{int(u):08x}" for u in nf4.midpoints().astype(np.float32).view(np.uint32))
    r = subprocess.run([str(exe)], input=mids, capture_output=True, text=True, timeout=600)
    print(r.stdout)
    assert r.returncode == 0, r.stdout + r.stderr
    assert " 0 mismatches" in r.stdout
