"""Pins of the oracle's storage rounding and of the one-byte gradient codec
(Section 3: the projected gradient sent as a signed log clipped to +-127; the
linear int8 code of the workloads). Rounding is checked by brute force against
the neighbouring representable values and against library conversions; the
codec exhaustively over all 255 codes."""
import math

import numpy as np
import pytest
import torch

import oracle


def bf16_value(bits: int) -> float:
    return float(np.array([bits << 16], dtype=np.uint32).view(np.float32)[0])


def test_bf16_rounding_is_nearest_with_ties_to_even(orc):
    rng = np.random.Generator(np.random.PCG64(21))
    xs = list(rng.standard_normal(3000) * 10.0 ** rng.integers(-40, 38, size=3000))
    xs += [2.0 ** -133, 2.0 ** -134, 3 * 2.0 ** -135, 2.0 ** -126 * 1.00390625]
    for x in xs:
        b = orc.round_bf16(x)
        r = bf16_value(b)
        lo, hi = bf16_value((b - 1) & 0xFFFF), bf16_value((b + 1) & 0xFFFF)
        d = abs(x - r)
        for nb in (lo, hi):
            if math.isfinite(nb) and (nb > 0) == (r > 0) and nb != 0:
                dn = abs(x - nb)
                assert d < dn or (d == dn and (b & 1) == 0), (x, b)


def test_bf16_ties_go_to_even(orc):
    one = 1.0
    ulp = 2.0 ** -7
    assert orc.round_bf16(one + ulp / 2) == 0x3F80          # tie -> even (1.0)
    assert orc.round_bf16(one + 3 * ulp / 2) == 0x3F82      # tie -> even (1+2ulp)
    assert orc.round_bf16(one + ulp / 2 + 2.0 ** -40) == 0x3F81  # past the tie
    assert orc.round_bf16(-(one + ulp / 2)) == 0xBF80
    assert orc.round_bf16(3.4e38) == 0x7F80                  # overflow to inf
    assert orc.round_bf16(0.0) == 0 and orc.round_bf16(-0.0) == 0x8000


def test_bf16_rounding_matches_torch_on_fp32_inputs(orc):
    """For values representable in fp32 a direct rounding equals torch's
    fp32 -> bf16 conversion (RNE)."""
    rng = np.random.Generator(np.random.PCG64(22))
    f = (rng.standard_normal(20000) * 10.0 ** rng.integers(-30, 30, size=20000)).astype(np.float32)
    want = torch.from_numpy(f).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = np.array([orc.round_bf16(float(v)) for v in f], dtype=np.uint16)
    assert np.array_equal(got, want)


def test_bf16_direct_rounding_differs_from_double_rounding(orc):
    """A value just above a bf16 tie whose fp32 rounding lands on the tie:
    direct rounding goes up, rounding through fp32 would go to even."""
    x = 1.0 + 2.0 ** -8 + 2.0 ** -30
    assert np.float32(x) == np.float32(1.0 + 2.0 ** -8)
    assert orc.round_bf16(x) == 0x3F81


def test_f32_rounding_matches_numpy(orc):
    rng = np.random.Generator(np.random.PCG64(23))
    for x in rng.standard_normal(2000) * 10.0 ** rng.integers(-45, 38, size=2000):
        assert np.float32(orc.round_f32(x)) == np.float64(x).astype(np.float32)


# ---- codec ---------------------------------------------------------------

ALL_Q = np.arange(-127, 128, dtype=np.int8)


@pytest.mark.parametrize("scale", [1.0 / 127.0, 0.25, 3.0e-3, 17.0])
def test_linear_round_trip_exhaustive(orc, scale):
    g = orc.dequantize(ALL_Q, oracle.LINEAR, scale)
    assert np.array_equal(orc.quantize(g, oracle.LINEAR, scale), ALL_Q)
    assert np.all(np.diff(g) > 0)


@pytest.mark.parametrize("alpha", [oracle.LOG2_ALPHA, 1.5, 4.0, 20.0])
def test_signed_log_round_trip_exhaustive(orc, alpha):
    g = orc.dequantize(ALL_Q, oracle.SIGNED_LOG, alpha=alpha)
    assert np.array_equal(orc.quantize(g, oracle.SIGNED_LOG, alpha=alpha), ALL_Q)
    assert np.all(np.sign(g) == np.sign(ALL_Q.astype(np.float64)))
    assert np.all(np.diff(g) > 0)


def test_linear_error_bound_and_monotone(orc):
    scale = 1.0 / 127.0
    g = np.linspace(-1.0, 1.0, 200001).astype(np.float32)
    q = orc.quantize(g, oracle.LINEAR, scale)
    back = orc.dequantize(q, oracle.LINEAR, scale).astype(np.float64)
    assert np.max(np.abs(back - g)) <= scale / 2 * (1 + 1e-6)
    assert np.all(np.diff(q.astype(np.int32)) >= 0)


def test_linear_ties_to_even_and_clipping(orc):
    q = orc.quantize(np.array([0.125, 0.375, 0.625, -0.625, 1e30, -np.inf, np.inf],
                              dtype=np.float32), oracle.LINEAR, 0.25)
    assert list(q) == [0, 2, 2, -2, 127, -127, 127]


def test_signed_log_closed_form(orc):
    """With the default base-2 log, g = 2^k - 1 codes to k; the sign is kept;
    zero maps to 0; the largest fp32 magnitudes clip to +-127; code 127
    decodes to ~2^127 - 1, still finite in fp32 (alpha is an fp32 value)."""
    ks = np.arange(0, 127)
    g = (2.0 ** ks.astype(np.float64) - 1.0).astype(np.float32)
    assert np.array_equal(orc.quantize(g, oracle.SIGNED_LOG), ks.astype(np.int8))
    assert np.array_equal(orc.quantize(-g, oracle.SIGNED_LOG), (-ks).astype(np.int8))
    assert list(orc.quantize(np.array([0.0, -0.0, 3.4e38, -np.inf], dtype=np.float32),
                             oracle.SIGNED_LOG)) == [0, 0, 127, -127]
    top = orc.dequantize(np.array([127, -127], dtype=np.int8), oracle.SIGNED_LOG)
    assert np.isfinite(top[0]) and top[0] == pytest.approx(2.0 ** 127, rel=1e-5)
    assert top[1] == -top[0]
    # a natural log scaled by alpha: alpha * ln(1 + |g|) = 10 for g = e - 1
    assert orc.quantize(np.array([math.e - 1], dtype=np.float32), oracle.SIGNED_LOG,
                        alpha=10.0)[0] == 10


def qmax_brute(alpha):
    """The largest k <= 127 with fl32(expm1(k / alpha)) finite, from numpy's
    float32 conversion."""
    best = 0
    for k in range(1, 128):
        with np.errstate(over="ignore"):
            if np.isfinite(np.float32(np.expm1(k / np.float64(np.float32(alpha))))):
                best = k
    return best


@pytest.mark.parametrize("alpha", [1.0, 0.5, 1.43, 1.4314, 1.44, oracle.LOG2_ALPHA, 0.02])
def test_signed_log_clip_where_fp32_ends(orc, alpha):
    """The code's range is +-127 or, below alpha ~1.4314, the largest code
    that still decodes to a finite fp32 (the natural log, alpha = 1: 88)."""
    qmax = orc.signed_log_qmax(alpha)
    assert qmax == qmax_brute(alpha)
    if alpha == 1.0:
        assert qmax == 88
    if alpha >= 1.44:
        assert qmax == 127
    codes = np.arange(-qmax, qmax + 1, dtype=np.int8)
    g = orc.dequantize(codes, oracle.SIGNED_LOG, alpha=alpha)
    assert np.all(np.isfinite(g)) and np.all(np.diff(g) > 0)
    assert np.array_equal(orc.quantize(g, oracle.SIGNED_LOG, alpha=alpha), codes)
    big = np.array([3.4e38, -np.inf, 1e30], dtype=np.float32)
    q = orc.quantize(big, oracle.SIGNED_LOG, alpha=alpha)
    assert q[0] == qmax and q[1] == -qmax
    if qmax < 127:
        with pytest.raises(oracle.OracleError):
            orc.dequantize(np.array([qmax + 1], dtype=np.int8), oracle.SIGNED_LOG, alpha=alpha)


def test_signed_log_natural_log_closed_form(orc):
    """alpha = 1: g = e^k - 1 codes to k (the literal natural-log reading)."""
    ks = np.arange(0, 60)
    g = np.expm1(ks.astype(np.float64)).astype(np.float32)
    assert np.array_equal(orc.quantize(g, oracle.SIGNED_LOG, alpha=1.0), ks.astype(np.int8))


def test_codec_rejects_bad_input(orc):
    with pytest.raises(oracle.OracleError):
        orc.quantize(np.array([np.nan], dtype=np.float32))
    with pytest.raises(oracle.OracleError):
        orc.dequantize(np.array([-128], dtype=np.int8))
    with pytest.raises(oracle.OracleError):
        orc.quantize(np.array([1.0], dtype=np.float32), oracle.LINEAR, 0.0)
    with pytest.raises(oracle.OracleError):
        orc.quantize(np.array([1.0], dtype=np.float32), oracle.SIGNED_LOG, alpha=-1.0)
    with pytest.raises(oracle.OracleError):   # even code 1 would decode past fp32
        orc.quantize(np.array([1.0], dtype=np.float32), oracle.SIGNED_LOG, alpha=1e-3)


def test_coefficient_sign_and_value(orc):
    """The apply loop perturbs with weight -grad * lr: positive code and
    positive lr give a negative weight equal to fl32(-lr * g~)."""
    q = np.array([127, -127, 1, 0], dtype=np.int8)
    c = orc.coefficients(q, 1e-6)
    g = orc.dequantize(q)
    assert c[0] < 0 and c[1] > 0 and c[3] == 0
    assert np.array_equal(c, (-np.float64(1e-6).astype(np.float32).astype(np.float64) *
                              g.astype(np.float64)).astype(np.float32))
    with pytest.raises(oracle.OracleError):
        orc.coefficients(q, float("nan"))
