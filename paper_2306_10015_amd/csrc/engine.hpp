// engine.hpp — device-side building blocks of the seeded perturbation engine
// for gfx950 (MI355X): the Philox generator, the Gaussian transform and the
// storage conversions.
//
// z for (seed, tensor t, element e) is defined in include/mezo.h: Philox4x32-10
// with key = machine id and counter = (e >> 2, t, sample, step), then
// Box-Muller on 24-bit uniforms. The paper only requires an RNG that every
// machine can reset to the same seed and replay (Algorithm 1,
// PerturbParameters; Appendix B on reproducing noise across devices); a
// counter-based generator lets every lane compute its own elements' noise in
// registers, so z is never stored.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "engine_launch.hpp"
#include "records.hpp"

namespace mezo {

__device__ __forceinline__ void mul_wide(uint32_t m, uint32_t x, uint32_t& hi, uint32_t& lo)
{
    uint64_t p = uint64_t(m) * uint64_t(x);
    hi = uint32_t(p >> 32);
    lo = uint32_t(p);
}

// a ^ b ^ c in one gfx950 v_bitop3_b32 (truth table 0x96 = three-way xor).
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c)
{
    return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);
}

// Per-call values that are the same for every element of one tensor: the
// round-1 words that do not depend on the element, and the round-2 product
// of the (element-independent) word 0. All scalar.
struct SeedUniform {
    uint32_t y1;        // round-1 output word 1
    uint32_t kx;        // step ^ key1: folded into round-1 output word 2
    uint32_t r2_hi;     // round 2: high word of kMulA * y0
    uint32_t r2_lo;     // round 2: low  word of kMulA * y0 (= output word 3)
    uint32_t k0, k1;    // round-2 key
};

__device__ __forceinline__ SeedUniform seed_uniform(const SeedRec& r, uint32_t tensor_id)
{
    SeedUniform u;
    // Round 1 on counter (blk, t, sample, step) with key (key0, key1):
    //   word 0 = hi(kMulB*sample) ^ t ^ key0   (element-independent)
    //   word 1 = lo(kMulB*sample)              (element-independent)
    //   word 2 = hi(kMulA*blk) ^ step ^ key1   (per element)
    //   word 3 = lo(kMulA*blk)                 (per element, seed-independent)
    uint32_t y0 = r.mb_hi ^ tensor_id ^ r.key0;
    u.y1 = r.mb_lo;
    u.kx = r.step ^ r.key1;
    u.k0 = r.key0 + kWeylA;
    u.k1 = r.key1 + kWeylB;
    mul_wide(kMulA, y0, u.r2_hi, u.r2_lo);
    return u;
}

// Seed-independent part of round 1 for block blk: kMulA * blk.
struct BlockPre {
    uint32_t hi, lo;
};

__device__ __forceinline__ BlockPre block_pre(uint32_t blk)
{
    BlockPre b;
    mul_wide(kMulA, blk, b.hi, b.lo);
    return b;
}

// The four Philox4x32-10 output words of one block, from the hoisted round-1
// values: rounds 2..10 with the per-element products on the vector unit.
__device__ __forceinline__ void philox_words(const SeedUniform& u, BlockPre b, uint32_t& x0,
                                             uint32_t& x1, uint32_t& x2, uint32_t& x3)
{
    // end of round 1
    uint32_t y2 = b.hi ^ u.kx;
    uint32_t y3 = b.lo;
    // round 2 (key k0, k1): products kMulA*y0 (scalar, precomputed) and kMulB*y2
    uint32_t hb, lb;
    mul_wide(kMulB, y2, hb, lb);
    x0 = hb ^ u.y1 ^ u.k0;
    x1 = lb;
    x2 = u.r2_hi ^ y3 ^ u.k1;
    x3 = u.r2_lo;
    uint32_t k0 = u.k0, k1 = u.k1;
#pragma unroll
    for (int round = 3; round <= 10; ++round) {
        k0 += kWeylA;
        k1 += kWeylB;
        uint32_t ha, la;
        mul_wide(kMulA, x0, ha, la);
        mul_wide(kMulB, x2, hb, lb);
        const uint32_t n0 = xor3(hb, x1, k0);
        const uint32_t n2 = xor3(ha, x3, k1);
        x0 = n0;
        x1 = lb;
        x2 = n2;
        x3 = la;
    }
}

// ---- Box-Muller -----------------------------------------------------------
// Box & Muller (1958). u1 = ((w_a >> 8) + 1) 2^-24 in (0, 1] and
// u2 = (w_b >> 8) 2^-24 in [0, 1) are exact in fp32. v_log_f32 is log2, so
// sqrt(-2 ln u1) = sqrt(2 ln 2) sqrt(-log2 u1); v_sin_f32 / v_cos_f32 take
// revolutions, so sin(2 pi u2) needs no multiply by 2 pi.
//
// gauss4_unit returns z / sqrt(2 ln 2): the constant factor is left to the
// caller, which folds it into the record's coefficient (one multiply per
// record on the host instead of two per Gaussian pair on the device).
struct Z4 {
    float z0, z1, z2, z3;
};

// sqrt(2 ln 2): z = kZScale * (the unit-scaled value below).
constexpr float kZScale = 1.17741002251547469101f;

__device__ __forceinline__ void box_muller_pair_unit(uint32_t wa, uint32_t wb, float& zc, float& zs)
{
    constexpr float kTwoM24 = 0x1p-24f;
    // (t + 1) 2^-24 as one fma: t < 2^24, so the product, the sum and the
    // result are exact.
    const float u1 = __builtin_fmaf(float(wa >> 8), kTwoM24, kTwoM24);
    const float u2 = float(wb >> 8) * kTwoM24;
    const float r = __builtin_amdgcn_sqrtf(-__builtin_amdgcn_logf(u1));
    zc = r * __builtin_amdgcn_cosf(u2);
    zs = r * __builtin_amdgcn_sinf(u2);
}

// acc_c += c z_c and acc_s += c z_s for one pair, with c the record's
// coefficient (which carries sqrt(2 ln 2)): c r is formed once and scales
// cos and sin inside the two fmas, so the pair costs one multiply.
__device__ __forceinline__ void box_muller_pair_acc(uint32_t wa, uint32_t wb, float c, float& acc_c, float& acc_s)
{
    constexpr float kTwoM24 = 0x1p-24f;
    const float u1 = __builtin_fmaf(float(wa >> 8), kTwoM24, kTwoM24);
    const float u2 = float(wb >> 8) * kTwoM24;
    const float cr = c * __builtin_amdgcn_sqrtf(-__builtin_amdgcn_logf(u1));
    acc_c = __builtin_fmaf(cr, __builtin_amdgcn_cosf(u2), acc_c);
    acc_s = __builtin_fmaf(cr, __builtin_amdgcn_sinf(u2), acc_s);
}

__device__ __forceinline__ Z4 gauss4_unit(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3)
{
    Z4 z;
    box_muller_pair_unit(w0, w1, z.z0, z.z1);
    box_muller_pair_unit(w2, w3, z.z2, z.z3);
    return z;
}

// The four Gaussians themselves (inspection path).
__device__ __forceinline__ Z4 gauss4(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3)
{
    Z4 z = gauss4_unit(w0, w1, w2, w3);
    z.z0 *= kZScale;
    z.z1 *= kZScale;
    z.z2 *= kZScale;
    z.z3 *= kZScale;
    return z;
}

// ---- portable Box-Muller ----------------------------------------------------
// The same Gaussian from binary32 +, -, *, fma, correctly rounded / and sqrt
// and exact scalings only, so that any IEEE device (a CPU included) computes
// it bit for bit (Appendix B: identical noise on every machine). -ln u1 comes
// from 2 atanh((m-1)/(m+1)) after an exact reduction of u1 to m 2^e with m in
// [sqrt(1/2), sqrt(2)); sin and cos of 2 pi u2 from the eighth of a turn that
// u2 falls in and Taylor polynomials on [0, pi/4] (coefficients 1/k! rounded
// to binary32). Division and sqrt are correctly rounded (below), as IEEE
// 754 requires of / and sqrt.

// n / d correctly rounded for normal n, d with a normal quotient and no
// overflow in the steps (the NF4 quantizer's 1 / m for a block maximum m in
// [2^-64, 2^64]): the reciprocal from v_rcp_f32 refined once, then two
// residual corrections of the quotient — the general sequence without its
// operand scaling and special-value fix-up, which only act outside that range.
__device__ __forceinline__ float div_rn_normal(float n, float d)
{
    float y = __builtin_amdgcn_rcpf(d);
    y = __builtin_fmaf(__builtin_fmaf(-d, y, 1.0f), y, y);
    float q = n * y;
    q = __builtin_fmaf(__builtin_fmaf(-d, q, n), y, q);
    return __builtin_fmaf(__builtin_fmaf(-d, q, n), y, q);
}

// sqrt(x) correctly rounded for x = 0 and normal x >= 2^-96 (here x = 0 or
// x in [2^-23, 34]): v_sqrt_f32, then the neighbour below or above replaces
// it when the residual shows it is nearer. At x = 0 the neighbour below is a
// NaN and the one above squares to 0, so 0 stays.
__device__ __forceinline__ float sqrt_rn_normal(float x)
{
    const float s = __builtin_amdgcn_sqrtf(x);
    const float lo = __uint_as_float(__float_as_uint(s) - 1u);
    const float hi = __uint_as_float(__float_as_uint(s) + 1u);
    float r = s;
    if (__builtin_fmaf(-lo, s, x) <= 0.0f) r = lo;
    if (__builtin_fmaf(-hi, s, x) > 0.0f) r = hi;
    return r;
}

// (m - 1) / (m + 1) correctly rounded for the m of the transform below: the
// reciprocal from v_rcp_f32 refined once, then one residual correction of the
// quotient (Markstein's scheme). That this rounds correctly for every m the
// transform meets (one per value of u1) is checked exhaustively: the GPU's z
// is bit-identical to the oracle's, which divides with IEEE /, over all 2^24
// values of u1.
__device__ __forceinline__ float div_rn_transform(float n, float d)
{
    float y = __builtin_amdgcn_rcpf(d);
    y = __builtin_fmaf(__builtin_fmaf(-d, y, 1.0f), y, y);
    const float q = n * y;
    return __builtin_fmaf(__builtin_fmaf(-d, q, n), y, q);
}

__device__ __forceinline__ void box_muller_pair_portable(uint32_t wa, uint32_t wb, float& zc, float& zs)
{
    // u1 = n1 2^-24 (n1 >= 1) = m 2^(e - 24) with m in [sqrt(1/2), sqrt(2)):
    // float(n1) is exact (n1 <= 2^24), and so are its mantissa mp in [1/2, 1)
    // and exponent ep (n1 = mp 2^ep); m is mp, or 2 mp below fl32(sqrt 2) / 2
    const float fn = float((wa >> 8) + 1u);
    const float mp = __builtin_amdgcn_frexp_mantf(fn);
    const int ep = __builtin_amdgcn_frexp_expf(fn);
    const bool upper = mp >= 0x1.6a09e6p-1f;                // fl32(sqrt 2) / 2
    const float m = upper ? mp : mp + mp;
    const int e = upper ? ep : ep - 1;
    const float f = m - 1.0f;                               // exact
    const float s = div_rn_transform(f, f + 2.0f);
    const float s2 = s * s;
    float p = __builtin_fmaf(s2, 0x1.c71c72p-4f, 0x1.24924ap-3f);  // 1/9, 1/7
    p = __builtin_fmaf(s2, p, 0x1.99999ap-3f);              // 1/5
    p = __builtin_fmaf(s2, p, 0x1.555556p-2f);              // 1/3
    p = __builtin_fmaf(s2, p, 1.0f);
    // ln m = fl32((s + s) p) and ln u1 = fl32((e - 24) fl32(ln 2) + ln m), each
    // carried here times -2, which is exact: a scaling by -2 changes no rounding
    const float m2ln_m = (s * -4.0f) * p;
    const float m2ln_u1 = __builtin_fmaf(float(e - 24), -0x1.62e430p+0f, m2ln_m);
    const float r = sqrt_rn_normal(m2ln_u1);            // sqrt(-2 ln u1)

    // u2 = t 2^-24 with t = wb >> 8: the octant q = floor(8 u2) is t's top
    // three bits; x = 8 u2 - q, or 1 - x in odd octants, is y = yl 2^-21 with
    // yl the low 21 bits of t or 2^21 minus them (exact, in integers); and
    // a = fl32(y fl32(pi/4)) = fl32(yl K), K = fl32(pi/4) 2^-21, since a power
    // of two scaling changes no rounding here
    const uint32_t q = wb >> 29;                            // octant
    const uint32_t tl = (wb >> 8) & 0x1FFFFFu;
    const uint32_t yl = (q & 1u) ? 0x200000u - tl : tl;     // [0, 2^21]
    const float a = float(yl) * 0x1.921fb6p-22f;            // fl32(pi/4) 2^-21
    const float a2 = a * a;
    float sn = __builtin_fmaf(a2, 0x1.71de3ap-19f, -0x1.a01a02p-13f);  // 1/9!, -1/7!
    sn = __builtin_fmaf(a2, sn, 0x1.111112p-7f);            // 1/5!
    sn = __builtin_fmaf(a2, sn, -0x1.555556p-3f);           // -1/3!
    sn = __builtin_fmaf(a2, sn, 1.0f);
    sn = a * sn;
    float cs = __builtin_fmaf(a2, -0x1.27e4fcp-22f, 0x1.a01a02p-16f);  // -1/10!, 1/8!
    cs = __builtin_fmaf(a2, cs, -0x1.6c16c2p-10f);          // -1/6!
    cs = __builtin_fmaf(a2, cs, 0x1.555556p-5f);            // 1/4!
    cs = __builtin_fmaf(a2, cs, -0.5f);                     // -1/2!
    cs = __builtin_fmaf(a2, cs, 1.0f);
    // angle = q pi/4 + a for even q, (q + 1) pi/4 - a for odd q
    const bool swap = (0x66u >> q) & 1u;                    // octants 1, 2, 5, 6
    const bool neg_cos = (0x3Cu >> q) & 1u;                 // octants 2..5
    const bool neg_sin = (q >> 2) & 1u;                     // octants 4..7
    float c0 = swap ? sn : cs;
    float s0 = swap ? cs : sn;
    if (neg_cos) c0 = -c0;
    if (neg_sin) s0 = -s0;
    zc = r * c0;
    zs = r * s0;
}

__device__ __forceinline__ Z4 gauss4_portable(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3)
{
    Z4 z;
    box_muller_pair_portable(w0, w1, z.z0, z.z1);
    box_muller_pair_portable(w2, w3, z.z2, z.z3);
    return z;
}

// acc_j += c z_j for the four Gaussians of one Philox block. Portable mode:
// the portable z, then fma(c, z, acc) as its definition states. Fast mode: c
// carries sqrt(2 ln 2), and each pair forms c r once (box_muller_pair_acc).
template <bool kPortable>
__device__ __forceinline__ void accumulate4(float c, uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3,
                                            float& a0, float& a1, float& a2, float& a3)
{
    if constexpr (kPortable) {
        const Z4 z = gauss4_portable(w0, w1, w2, w3);
        a0 = __builtin_fmaf(c, z.z0, a0);
        a1 = __builtin_fmaf(c, z.z1, a1);
        a2 = __builtin_fmaf(c, z.z2, a2);
        a3 = __builtin_fmaf(c, z.z3, a3);
    } else {
        box_muller_pair_acc(w0, w1, c, a0, a1);
        box_muller_pair_acc(w2, w3, c, a2, a3);
    }
}

// acc_j = c z_j for the four Gaussians of one block in fast mode (a step's
// first record: no accumulator to clear first). The product differs from
// fma(c, z, +0) only in the sign of a zero product, which changes theta + acc
// only for theta = -0 (a -0 result where the accumulator's +0 gives +0).
__device__ __forceinline__ void assign4_fast(float c, uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3,
                                             float& a0, float& a1, float& a2, float& a3)
{
    constexpr float kTwoM24 = 0x1p-24f;
    const float u1a = __builtin_fmaf(float(w0 >> 8), kTwoM24, kTwoM24);
    const float u2a = float(w1 >> 8) * kTwoM24;
    const float cra = c * __builtin_amdgcn_sqrtf(-__builtin_amdgcn_logf(u1a));
    a0 = cra * __builtin_amdgcn_cosf(u2a);
    a1 = cra * __builtin_amdgcn_sinf(u2a);
    const float u1b = __builtin_fmaf(float(w2 >> 8), kTwoM24, kTwoM24);
    const float u2b = float(w3 >> 8) * kTwoM24;
    const float crb = c * __builtin_amdgcn_sqrtf(-__builtin_amdgcn_logf(u1b));
    a2 = crb * __builtin_amdgcn_cosf(u2b);
    a3 = crb * __builtin_amdgcn_sinf(u2b);
}

// Record r of a launch: from the kernel arguments (kInline) or the staged
// device buffer. Either way a wave-uniform address: the words go to SGPRs.
template <bool kInline>
__device__ __forceinline__ const SeedRec& rec_at(const EngineArgs& a, uint32_t r)
{
    if constexpr (kInline)
        return a.inl[r];
    else
        return a.ext[r];
}

// ---- storage conversions ---------------------------------------------------

__device__ __forceinline__ float bf16_lo(uint32_t packed) { return __uint_as_float(packed << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t packed) { return __uint_as_float(packed & 0xFFFF0000u); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two fp32 -> two bf16 (round to nearest even, one v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi)
{
    f32x2_t v = {lo, hi};
    bf16x2_t b = __builtin_convertvector(v, bf16x2_t);
    return __builtin_bit_cast(uint32_t, b);
}

__device__ __forceinline__ uint16_t to_bf16(float x)
{
    __bf16 b = static_cast<__bf16>(x);
    return __builtin_bit_cast(uint16_t, b);
}

}  // namespace mezo
