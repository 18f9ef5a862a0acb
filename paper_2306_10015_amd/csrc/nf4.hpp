// nf4.hpp — the 4-bit NormalFloat storage of the 4-bit forward-only variant
// (Section 3: weights dequantized before the noise is added and quantized
// again afterwards, in QLoRA's 4-bit format, which the paper cites there).
//
// The 16 values are QLoRA's NF4: quantiles of N(0, 1) for an asymmetric pair
// of halves (8 positive, 7 negative, an exact zero), scaled to [-1, 1],
// rounded to fp32. Quantizing x in [-1, 1] picks the nearest value, a tie
// going to the lower code: code = number of midpoints m_i = fl32((v_i +
// v_{i+1}) / 2) strictly below x.
//
// Fast exact lookup: x maps to one of a few more than 128 bins by a
// monotone function b(x), and no bin holds two midpoints (the values are more
// than 1/64 apart). For x in bin b, every midpoint in a lower bin is below x
// and every midpoint in a higher bin above it, so code = (midpoints in bins
// below b) + (x > the midpoint in bin b, if any). The tables are built at
// compile time from the same b() the kernels evaluate. Two bin functions:
//
// - kNF4Table, 128 bins: b(x) = floor(fl32(64 x + 64)) clamped to [0, 127]
//   (fma rounds 64 x + 64 once, exactly as the double expression below
//   rounded to float does); used by the kernel that applies long record
//   lists.
// - kNF4RoundTable, 129 bins: b(x) = the integer nearest to 64 x + 64 (ties to
//   even), which one fma gives directly: t = fl32(64 x + kNF4BinMagic),
//   kNF4BinMagic = 1.5 * 2^23 + 64, lies in [2^23, 2^24) where floats are 1
//   apart, so t is 64 x + 64 rounded once to the nearest integer plus 1.5 *
//   2^23, and the bit pattern of t is kNF4BinBase + b. For |x| <= 1 + 2^-23
//   (every x of a block whose maximum has a normal reciprocal), b is in
//   [0, 128] with no clamp; used by the kernel for one- and two-record calls
//   and by the standalone quantization.
#pragma once

#include <stdint.h>

#include "records.hpp"

namespace mezo {

constexpr int kNF4Codes = 16;
constexpr uint32_t kNF4ZeroCode = 7;
constexpr int kNF4Bins = 128;
constexpr int kNF4RoundBins = 129;
constexpr float kNF4BinMagic = 12582976.0f;      // 1.5 * 2^23 + 64
constexpr uint32_t kNF4BinBase = 0x4B400000u;    // bit pattern of 1.5 * 2^23
constexpr int kNF4Pairs = 256;                   // byte -> the values of its two codes

constexpr float kNF4Values[kNF4Codes] = {
    -0x1.000000p+0f, -0x1.647362p-1f, -0x1.0cd65cp-1f, -0x1.94653cp-2f,
    -0x1.234496p-2f, -0x1.7a6a7ap-3f, -0x1.74f0d2p-4f, 0.0f,
    0x1.45f602p-4f,  0x1.4995bep-3f,  0x1.f809b4p-3f,  0x1.5a066cp-2f,
    0x1.c3496ap-2f,  0x1.200f52p-1f,  0x1.722760p-1f,  0x1.000000p+0f,
};

constexpr float nf4_midpoint(int i)
{
    return static_cast<float>((double(kNF4Values[i]) + double(kNF4Values[i + 1])) * 0.5);
}

// b(x) as the kernels compute it: fma(x, 64, 64), truncated to int, clamped.
constexpr int nf4_bin_of(float x)
{
    const float t = static_cast<float>(double(x) * 64.0 + 64.0);
    const int b = static_cast<int>(t);
    return b < 0 ? 0 : (b > kNF4Bins - 1 ? kNF4Bins - 1 : b);
}

// The round-to-nearest bin function: 64 x + 64 (exact in double for a float
// x) rounded to the nearest integer, ties to even, clamped to [0, 128].
constexpr int nf4_round_bin_of(float x)
{
    const double t = double(x) * 64.0 + 64.0;
    if (t <= 0.0) return 0;
    if (t >= double(kNF4RoundBins - 1)) return kNF4RoundBins - 1;
    const int f = static_cast<int>(t);  // floor, t > 0
    const double d = t - double(f);
    return d > 0.5 ? f + 1 : (d < 0.5 ? f : (f % 2 == 0 ? f : f + 1));
}

// One bin: its midpoint (+inf if none), the code below it and the values of
// that code and the next.
struct alignas(16) NF4Bin {
    float mid;
    uint32_t lo;
    float v_lo;
    float v_hi;
};

template <int kBins>
struct NF4Table {
    NF4Bin bin[kBins];
    bool ok;  // no bin holds two midpoints
};

template <int kBins, int (*kBinOf)(float)>
constexpr NF4Table<kBins> make_nf4_table()
{
    NF4Table<kBins> t{};
    t.ok = true;
    for (int b = 0; b < kBins; ++b) {
        uint32_t lo = 0;
        int in_bin = 0;
        float mid = __builtin_huge_valf();
        for (int i = 0; i < kNF4Codes - 1; ++i) {
            const int mb = kBinOf(nf4_midpoint(i));
            if (mb < b) ++lo;
            if (mb == b) {
                mid = nf4_midpoint(i);
                ++in_bin;
            }
        }
        if (in_bin > 1) t.ok = false;
        t.bin[b].mid = mid;
        t.bin[b].lo = lo;
        t.bin[b].v_lo = kNF4Values[lo];
        t.bin[b].v_hi = kNF4Values[lo + 1 < kNF4Codes ? lo + 1 : lo];
    }
    return t;
}

constexpr NF4Table<kNF4Bins> kNF4Table = make_nf4_table<kNF4Bins, nf4_bin_of>();
static_assert(kNF4Table.ok, "two NF4 midpoints share a bin");
static_assert(nf4_bin_of(-1.0f) == 0 && nf4_bin_of(1.0f) == kNF4Bins - 1, "bin range");

constexpr NF4Table<kNF4RoundBins> kNF4RoundTable = make_nf4_table<kNF4RoundBins, nf4_round_bin_of>();
static_assert(kNF4RoundTable.ok, "two NF4 midpoints share a bin");
// the extremes of a block with a normal reciprocal: |x| <= 1 + 2^-23
static_assert(nf4_round_bin_of(-1.00000012f) == 0 && nf4_round_bin_of(1.00000012f) == kNF4RoundBins - 1,
              "bin range");
static_assert(__builtin_bit_cast(uint32_t, 12582912.0f) == kNF4BinBase, "magic base");
static_assert(kNF4BinMagic == 12582912.0f + 64.0f, "magic constant");

}  // namespace mezo
