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
// Fast exact lookup: x maps to one of 128 bins by b(x) = floor(fl32(64 x +
// 64)) clamped to [0, 127], a monotone function of x, and no bin holds two
// midpoints (the values are more than 1/64 apart). For x in bin b, every
// midpoint in a lower bin is below x and every midpoint in a higher bin above
// it, so code = (midpoints in bins below b) + (x > the midpoint in bin b, if
// any). The table is built at compile time from the same b() the kernels
// evaluate (fma rounds 64 x + 64 once, exactly as the double expression below
// rounded to float does).
#pragma once

#include <stdint.h>

namespace mezo {

constexpr int kNF4Codes = 16;
constexpr uint32_t kNF4ZeroCode = 7;
constexpr int kNF4Block = 64;
constexpr int kNF4Bins = 128;

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

// One bin: its midpoint (+inf if none), the code below it and the values of
// that code and the next.
struct alignas(16) NF4Bin {
    float mid;
    uint32_t lo;
    float v_lo;
    float v_hi;
};

struct NF4Table {
    NF4Bin bin[kNF4Bins];
    bool ok;  // no bin holds two midpoints
};

constexpr NF4Table make_nf4_table()
{
    NF4Table t{};
    t.ok = true;
    for (int b = 0; b < kNF4Bins; ++b) {
        uint32_t lo = 0;
        int in_bin = 0;
        float mid = __builtin_huge_valf();
        for (int i = 0; i < kNF4Codes - 1; ++i) {
            const int mb = nf4_bin_of(nf4_midpoint(i));
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

constexpr NF4Table kNF4Table = make_nf4_table();
static_assert(kNF4Table.ok, "two NF4 midpoints share a bin");
static_assert(nf4_bin_of(-1.0f) == 0 && nf4_bin_of(1.0f) == kNF4Bins - 1, "bin range");

}  // namespace mezo
