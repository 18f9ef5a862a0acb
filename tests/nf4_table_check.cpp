// nf4_table_check.cpp — TEST INFRASTRUCTURE ONLY: the two bin tables of
// nf4.hpp and the lookup arithmetic of the NF4 kernels (nf4_ops.hpp) replayed
// on the host: the 128-bin floor table over every float x with |x| <= 1 +
// 2^-22 and special values; the 129-bin round-to-nearest table with the
// short path's fast lookup over every such x (its domain: there |x| <= 1 +
// 2^-23) and its general lookup over those and special values.
// Each code is compared with the number of midpoints strictly below x, the
// midpoints being read from stdin (the oracle's, 15 floats as hex bit
// patterns). Prints the number of mismatches and exits 0 when there are none.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>

#include "nf4.hpp"

static uint32_t bits(float x)
{
    uint32_t u;
    std::memcpy(&u, &x, 4);
    return u;
}

static float from_bits(uint32_t u)
{
    float x;
    std::memcpy(&x, &u, 4);
    return x;
}

using mezo::kNF4Bins;
using mezo::kNF4RoundBins;
using mezo::kNF4RoundTable;
using mezo::kNF4Table;

// floor table: b = trunc(fl32(64 x + 64)) clamped to [0, 127]
static uint32_t code_floor(float x)
{
    const float t = std::fmaf(x, 64.0f, 64.0f);
    int b = t == t ? int(t) : 0;  // the hardware conversion takes NaN to 0
    if (!(t > -2147483648.0f)) b = 0;
    if (!(t < 2147483648.0f) && t == t) b = kNF4Bins - 1;
    b = b < 0 ? 0 : (b > kNF4Bins - 1 ? kNF4Bins - 1 : b);
    const mezo::NF4Bin& e = kNF4Table.bin[b];
    return e.lo + (x > e.mid ? 1u : 0u);
}

// round-to-nearest table, fast lookup: t = fl32(64 x + magic) with one
// rounding; entry offset 16 (t - base)
static uint32_t code_fast(float x)
{
    const uint32_t t = bits(std::fmaf(x, 64.0f, mezo::kNF4BinMagic));
    const uint32_t off = (t << 4) - (mezo::kNF4BinBase << 4);
    if (off % 16 != 0 || off / 16 >= uint32_t(kNF4RoundBins)) return 99;  // would read past the table
    const mezo::NF4Bin& e = kNF4RoundTable.bin[off / 16];
    return e.lo + (x > e.mid ? 1u : 0u);
}

// round-to-nearest table, general lookup: NaN to -2, the bin clamped
static uint32_t code_general(float x)
{
    const float xs = x == x ? x : -2.0f;
    const int k = int(bits(std::fmaf(xs, 64.0f, mezo::kNF4BinMagic))) - int(mezo::kNF4BinBase);
    const mezo::NF4Bin& e = kNF4RoundTable.bin[k < 0 ? 0 : (k > kNF4RoundBins - 1 ? kNF4RoundBins - 1 : k)];
    return e.lo + (x > e.mid ? 1u : 0u);
}

int main()
{
    float mid[15];
    for (int i = 0; i < 15; ++i) {
        unsigned u;
        if (std::scanf("%x", &u) != 1) return 2;
        mid[i] = from_bits(u);
    }
    const auto want = [&](float x) {
        uint32_t c = 0;
        for (int i = 0; i < 15; ++i) c += mid[i] < x ? 1u : 0u;
        return c;
    };
    unsigned long long bad = 0, n = 0;
    const uint32_t hi = bits(1.0f) + 2;  // 1 + 2^-22
    for (uint32_t s = 0; s < 2; ++s) {
        for (uint32_t m = 0; m <= hi; ++m) {
            const float x = from_bits(m | (s << 31));
            const uint32_t w = want(x);
            bad += code_floor(x) != w;
            bad += code_fast(x) != w;
            bad += code_general(x) != w;
            n += 3;
        }
    }
    // special and out-of-range values the general path meets
    const float special[] = {INFINITY, -INFINITY, NAN, 3.4e38f, -3.4e38f, 2.0f, -2.0f, 1e6f, -1e6f, 1.5e5f, -1.5e5f};
    for (float x : special) {
        const uint32_t w = x == x ? want(x) : 0u;  // NaN: no midpoint is below it
        bad += code_general(x) != w;
        bad += code_floor(x) != w;
        n += 2;
    }
    std::printf("%llu lookups, %llu mismatches\n", n, bad);
    return bad ? 1 : 0;
}
