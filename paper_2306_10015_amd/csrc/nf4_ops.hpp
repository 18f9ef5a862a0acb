// nf4_ops.hpp — device helpers of the 4-bit storage (the 4-bit forward-only
// variant of Section 3), shared by the NF4 engine kernel and the standalone
// conversions.
//
// A lane owns 8 consecutive elements (one dword of codes); the 8 lanes
// tid & ~7 .. tid | 7 own one 64-element block and share its absmax. Codes
// become values through a 16-entry table and values become codes through the
// 128-bin table of nf4.hpp. Calls of one or two records (where the per-element
// work around the noise weighs most) take the short path at the end of this
// file: a table of byte -> the values of its two codes, the 129-bin
// round-to-nearest table, and a shorter reciprocal; one-record calls with 16
// elements per lane (4 lanes per block).
#pragma once

#include "engine.hpp"
#include "nf4.hpp"
#include "stream_io.hpp"

namespace mezo {

struct NF4Lds {
    NF4Bin bin[kNF4Bins];
    float val[kNF4Codes];
};

__device__ __forceinline__ void nf4_lds_init(NF4Lds& s)
{
    if (threadIdx.x < kNF4Bins) s.bin[threadIdx.x] = kNF4Table.bin[threadIdx.x];
    if (threadIdx.x < kNF4Codes) s.val[threadIdx.x] = kNF4Values[threadIdx.x];
    __syncthreads();
}

// Whether any lane of the wave misses elements (valid != 0xFF; only waves
// that reach a tensor's end): a uniform test, so that the masking it guards
// stays a branch that every other wave skips instead of selects that every
// wave executes.
__device__ __forceinline__ bool partial_wave(uint32_t valid)
{
    return __builtin_amdgcn_ballot_w64(valid != 0xFFu) != 0;
}

// Which of a lane's 8 elements e0 .. e0 + 7 exist (bit j for element e0 + j).
__device__ __forceinline__ uint32_t nf4_valid(uint64_t e0, uint64_t numel)
{
    if (e0 >= numel) return 0u;
    if (e0 + 8 <= numel) return 0xFFu;
    return (1u << uint32_t(numel - e0)) - 1u;
}

// A lane's code dword and its block's absmax (zeros past the end). kFull:
// the lane's 8 elements are known to exist (a tile wholly inside its tensor).
template <bool kFull = false>
__device__ __forceinline__ void nf4_load(uint64_t codes, uint64_t absmax, uint64_t e0, uint64_t numel,
                                         uint32_t& packed, float& am)
{
    packed = 0u;
    am = 0.0f;
    if (!kFull && e0 >= numel) return;
    if (kFull || e0 + 8 <= numel) {
        packed = __builtin_nontemporal_load(reinterpret_cast<const MEZO_GLOBAL uint32_t*>(codes + e0 / 2));
    } else {
        const MEZO_GLOBAL uint8_t* b = reinterpret_cast<const MEZO_GLOBAL uint8_t*>(codes + e0 / 2);
#pragma unroll
        for (uint32_t k = 0; k < 4; ++k)
            if (e0 + 2 * k < numel) packed |= uint32_t(b[k]) << (8 * k);
    }
    am = reinterpret_cast<const gfloat_t*>(absmax)[e0 / kNF4Block];
}

template <bool kFull = false>
__device__ __forceinline__ void nf4_store(uint64_t codes, uint64_t absmax, uint64_t e0, uint64_t numel,
                                          uint32_t packed, float am)
{
    if (!kFull && e0 >= numel) return;
    if (kFull || e0 + 8 <= numel) {
        __builtin_nontemporal_store(packed, reinterpret_cast<MEZO_GLOBAL uint32_t*>(codes + e0 / 2));
    } else {
        MEZO_GLOBAL uint8_t* b = reinterpret_cast<MEZO_GLOBAL uint8_t*>(codes + e0 / 2);
#pragma unroll
        for (uint32_t k = 0; k < 4; ++k)
            if (e0 + 2 * k < numel) b[k] = uint8_t(packed >> (8 * k));
    }
    if ((threadIdx.x & 7u) == 0u) reinterpret_cast<gfloat_t*>(absmax)[e0 / kNF4Block] = am;
}

__device__ __forceinline__ void nf4_dequant(const NF4Lds& s, uint32_t packed, float am, uint32_t valid,
                                            float (&w)[8])
{
#pragma unroll
    for (int j = 0; j < 8; ++j) w[j] = s.val[(packed >> (4 * j)) & 15u] * am;
    if (partial_wave(valid)) {  // only waves that reach a tensor's end
#pragma unroll
        for (int j = 0; j < 8; ++j)
            if (!((valid >> j) & 1u)) w[j] = 0.0f;
    }
}

// max over the 8 lanes of a block (lanes 8i .. 8i + 7) of a value >= 0:
// swap neighbours, then pairs within each quad, then the two quads of each
// half-row (DPP quad_perm [1,0,3,2], quad_perm [2,3,0,1], row_half_mirror).
// Non-negative floats order like their bit patterns, so the maximum is taken
// on the integers.
__device__ __forceinline__ float max8(float m)
{
    uint32_t u = __float_as_uint(m);
    u = max(u, uint32_t(__builtin_amdgcn_update_dpp(0, int(u), 0xB1, 0xF, 0xF, false)));
    u = max(u, uint32_t(__builtin_amdgcn_update_dpp(0, int(u), 0x4E, 0xF, 0xF, false)));
    u = max(u, uint32_t(__builtin_amdgcn_update_dpp(0, int(u), 0x141, 0xF, 0xF, false)));
    return __uint_as_float(u);
}

// Nibbles of the packed codes that hold existing elements.
__device__ __forceinline__ uint32_t nf4_nibble_mask(uint32_t valid)
{
    const uint32_t k = __builtin_popcount(valid);  // valid is a run of low bits
    return k >= 8 ? 0xFFFFFFFFu : (1u << (4 * k)) - 1u;
}

// Quantize a block held by 8 lanes (w = 0 for elements that do not exist):
// a = max |w| over the block, r = 1 / a (correctly rounded; 0 for a = 0),
// code = nearest NF4 value to fl32(w * r), ties to the lower code. Returns the
// packed codes (0 for missing elements) and the new absmax; with kNext it also
// replaces w by the dequantized values fl32(v * a) the next step starts from
// (0 stays 0: x = 0 lies in a bin without a midpoint whose lower value is 0).
// Every lane of the wave must call it (the block maximum is exchanged across
// lanes).
template <bool kNext>
__device__ __forceinline__ void nf4_requant(const NF4Bin* bins, uint32_t valid, float (&w)[8], uint32_t& packed,
                                            float& am)
{
    float m = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) m = fmaxf(m, fabsf(w[j]));
    m = max8(m);
    const float r = m > 0.0f ? 1.0f / m : 0.0f;
    uint32_t p = 0u;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const float x = w[j] * r;
        int b = static_cast<int>(__builtin_fmaf(x, 64.0f, 64.0f));
        b = b < 0 ? 0 : (b > kNF4Bins - 1 ? kNF4Bins - 1 : b);
        const NF4Bin e = bins[b];
        const bool up = x > e.mid;
        if constexpr (kNext) w[j] = (up ? e.v_hi : e.v_lo) * m;
        p |= (e.lo + (up ? 1u : 0u)) << (4 * j);
    }
    packed = partial_wave(valid) ? p & nf4_nibble_mask(valid) : p;
    am = m;
}

// ---- the short path: calls of one or two records ---------------------------

// The LDS tables of the short path, laid out as one image of 257 rows of 16
// bytes that a workgroup copies from constant memory with one row per lane
// (and the last row by lane 0): the 129 round-to-nearest bins, then byte b ->
// the values of its two codes (b & 15, b >> 4).
struct NF4Pair {
    float v_lo, v_hi;
};
struct alignas(16) NF4ShortLds {
    NF4Bin bin[kNF4RoundBins];
    NF4Pair pair[kNF4Pairs];
};
static_assert(kThreads == kNF4Pairs && kThreads >= kNF4RoundBins, "one table entry per lane");
static_assert(sizeof(NF4ShortLds) == 16 * (kThreads + 1), "257 rows of 16 bytes");

constexpr NF4ShortLds make_nf4_short_image()
{
    NF4ShortLds s{};
    for (int b = 0; b < kNF4RoundBins; ++b) s.bin[b] = kNF4RoundTable.bin[b];
    for (int b = 0; b < kNF4Pairs; ++b) s.pair[b] = NF4Pair{kNF4Values[b & 15], kNF4Values[b >> 4]};
    return s;
}
constexpr NF4ShortLds kNF4ShortImage = make_nf4_short_image();

__device__ __forceinline__ void nf4_short_lds_init(NF4ShortLds& s)
{
    const u32x4_t* src = reinterpret_cast<const u32x4_t*>(&kNF4ShortImage);
    u32x4_t* dst = reinterpret_cast<u32x4_t*>(&s);
    dst[threadIdx.x] = src[threadIdx.x];
    if (threadIdx.x == 0) dst[kThreads] = src[kThreads];
    __syncthreads();
}

// Byte k of packed times 8, the LDS byte offset of its entry in the pair
// table: one shift with sub-dword (SDWA) selection of the byte.
template <int k>
__device__ __forceinline__ uint32_t byte_x8(uint32_t packed)
{
    uint32_t off;
    if constexpr (k == 0)
        asm("v_lshlrev_b32_sdwa %0, 3, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_0"
            : "=v"(off) : "v"(packed));
    else if constexpr (k == 1)
        asm("v_lshlrev_b32_sdwa %0, 3, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_1"
            : "=v"(off) : "v"(packed));
    else if constexpr (k == 2)
        asm("v_lshlrev_b32_sdwa %0, 3, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_2"
            : "=v"(off) : "v"(packed));
    else
        asm("v_lshlrev_b32_sdwa %0, 3, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_3"
            : "=v"(off) : "v"(packed));
    return off;
}

template <int k>
__device__ __forceinline__ float2 nf4_pair(const NF4ShortLds& s, uint32_t packed)
{
    return *reinterpret_cast<const float2*>(reinterpret_cast<const char*>(s.pair) + byte_x8<k>(packed));
}

// nf4_dequant through the pair table: each code byte fetches the values of
// its two codes at once.
__device__ __forceinline__ void nf4_dequant_pairs(const NF4ShortLds& s, uint32_t packed, float am, uint32_t valid,
                                                  float (&w)[8])
{
    const float2 p0 = nf4_pair<0>(s, packed);
    const float2 p1 = nf4_pair<1>(s, packed);
    const float2 p2 = nf4_pair<2>(s, packed);
    const float2 p3 = nf4_pair<3>(s, packed);
    w[0] = p0.x * am;
    w[1] = p0.y * am;
    w[2] = p1.x * am;
    w[3] = p1.y * am;
    w[4] = p2.x * am;
    w[5] = p2.y * am;
    w[6] = p3.x * am;
    w[7] = p3.y * am;
    if (partial_wave(valid)) {  // only waves that reach a tensor's end
#pragma unroll
        for (int j = 0; j < 8; ++j)
            if (!((valid >> j) & 1u)) w[j] = 0.0f;
    }
}

// ---- one-record calls: 16 elements per lane ----------------------------------
// A perturbation (one record) needs no accumulators, so a lane can own 16
// elements (4 Philox blocks, a quarter of an absmax block) within 64 VGPRs:
// 128-lane workgroups over the same 2048-element tiles, and the work paid per
// lane (tile addressing, the table copy, the block maximum across lanes, the
// reciprocal) spread over twice the elements.

constexpr int kSweepLanes = 128;  // lanes per workgroup of the one-record kernel
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef MEZO_GLOBAL u32x2_t gu32x2_t;

// Copy the short-path image to LDS with 128 lanes: rows lane and lane + 128,
// and the last row by lane 0.
__device__ __forceinline__ void nf4_sweep_lds_init(NF4ShortLds& s)
{
    const u32x4_t* src = reinterpret_cast<const u32x4_t*>(&kNF4ShortImage);
    u32x4_t* dst = reinterpret_cast<u32x4_t*>(&s);
    dst[threadIdx.x] = src[threadIdx.x];
    dst[threadIdx.x + kSweepLanes] = src[threadIdx.x + kSweepLanes];
    if (threadIdx.x == 0) dst[2 * kSweepLanes] = src[2 * kSweepLanes];
    __syncthreads();
}
static_assert(2 * kSweepLanes == kThreads, "the image is 2 x 128 rows plus one");

// Which of a lane's 16 elements e0 .. e0 + 15 exist (bit j for element e0 + j).
__device__ __forceinline__ uint32_t nf4_valid16(uint64_t e0, uint64_t numel)
{
    if (e0 >= numel) return 0u;
    if (e0 + 16 <= numel) return 0xFFFFu;
    return (1u << uint32_t(numel - e0)) - 1u;
}

__device__ __forceinline__ bool partial_wave16(uint32_t valid)
{
    return __builtin_amdgcn_ballot_w64(valid != 0xFFFFu) != 0;
}

// nf4_dequant_pairs for 16 elements: packed[0] holds elements 0..7, packed[1]
// elements 8..15.
__device__ __forceinline__ void nf4_dequant_pairs16(const NF4ShortLds& s, const uint32_t (&packed)[2], float am,
                                                    uint32_t valid, float (&w)[16])
{
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const float2 p0 = nf4_pair<0>(s, packed[h]);
        const float2 p1 = nf4_pair<1>(s, packed[h]);
        const float2 p2 = nf4_pair<2>(s, packed[h]);
        const float2 p3 = nf4_pair<3>(s, packed[h]);
        w[8 * h + 0] = p0.x * am;
        w[8 * h + 1] = p0.y * am;
        w[8 * h + 2] = p1.x * am;
        w[8 * h + 3] = p1.y * am;
        w[8 * h + 4] = p2.x * am;
        w[8 * h + 5] = p2.y * am;
        w[8 * h + 6] = p3.x * am;
        w[8 * h + 7] = p3.y * am;
    }
    if (partial_wave16(valid)) {  // only waves that reach a tensor's end
#pragma unroll
        for (int j = 0; j < 16; ++j)
            if (!((valid >> j) & 1u)) w[j] = 0.0f;
    }
}

// max over the 4 lanes of a block (one quad) of a value >= 0, on the integers
// as in max8.
__device__ __forceinline__ float max4(float m)
{
    uint32_t u = __float_as_uint(m);
    u = max(u, uint32_t(__builtin_amdgcn_update_dpp(0, int(u), 0xB1, 0xF, 0xF, false)));
    u = max(u, uint32_t(__builtin_amdgcn_update_dpp(0, int(u), 0x4E, 0xF, 0xF, false)));
    return __uint_as_float(u);
}

// (p << 4) | c as one v_lshl_or_b32 (left to itself the compiler splits a
// chain of these into separate shifts and three-way ors).
__device__ __forceinline__ uint32_t shl4_or(uint32_t p, uint32_t c)
{
    uint32_t r;
    asm("v_lshl_or_b32 %0, %1, 4, %2" : "=v"(r) : "v"(p), "v"(c));
    return r;
}

// Block maxima whose reciprocal takes the short sequence: [2^-64, 2^64].
constexpr uint32_t kRecipLo = 0x1F800000u;  // 2^-64
constexpr uint32_t kRecipHi = 0x5F800000u;  // 2^64

// nf4_requant on the round-to-nearest table. When every lane's block maximum
// a lies in [2^-64, 2^64] (the usual case), r = 1 / a comes from the
// correctly rounded division sequence without its operand scaling and
// special-value fix-up (which act only outside that range), every |x| <= 1 +
// 2^-23, and the bin's table offset is read off t = fl32(64 x + magic)
// directly. Otherwise (a = 0, tiny or huge blocks; x may be infinite or NaN)
// the wave takes the general division and clamps the bin to the table, a NaN
// x (0 * inf) taking the lowest bin like the comparisons it fails. Same
// result as nf4_requant either way. kExactRecip = false (the engine's fast
// mode) takes v_rcp_f32's reciprocal in the usual case, as
// nf4_requant_round16 does.
template <bool kNext, bool kExactRecip = true>
__device__ __forceinline__ void nf4_requant_round(const NF4Bin* bins, uint32_t valid, float (&w)[8],
                                                  uint32_t& packed, float& am)
{
    float m = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) m = fmaxf(m, fabsf(w[j]));
    m = max8(m);
    const bool usual = __float_as_uint(m) - kRecipLo <= kRecipHi - kRecipLo;
    const char* base = reinterpret_cast<const char*>(bins);
    // the codes enter p from the highest element down: p = (p << 4) | code
    // (the loops below run j = 7 .. 0)
    uint32_t p = 0u;
    const auto code = [&](int j, float x, uint32_t off) {
        if constexpr (kNext) {
            const NF4Bin e = *reinterpret_cast<const NF4Bin*>(base + off);
            const bool up = x > e.mid;
            w[j] = (up ? e.v_hi : e.v_lo) * m;
            const uint32_t c = e.lo + (up ? 1u : 0u);
            p = j == 7 ? c : shl4_or(p, c);
        } else {
            const float2 e = *reinterpret_cast<const float2*>(base + off);  // mid, lo
            const uint32_t c = __float_as_uint(e.y) + (x > e.x ? 1u : 0u);
            p = j == 7 ? c : shl4_or(p, c);
        }
    };
    if (__builtin_amdgcn_ballot_w64(!usual) == 0) {  // uniform
        const float r = kExactRecip ? div_rn_normal(1.0f, m) : __builtin_amdgcn_rcpf(m);
#pragma unroll
        for (int j = 7; j >= 0; --j) {
            const float x = w[j] * r;
            const uint32_t t = __float_as_uint(__builtin_fmaf(x, 64.0f, kNF4BinMagic));
            code(j, x, (t << 4) - (kNF4BinBase << 4));  // 16 (t - base) = 16 b
        }
    } else {
        const float r = m > 0.0f ? 1.0f / m : 0.0f;
#pragma unroll
        for (int j = 7; j >= 0; --j) {
            const float x = w[j] * r;
            const float xs = x == x ? x : -2.0f;
            const int k = int(__float_as_uint(__builtin_fmaf(xs, 64.0f, kNF4BinMagic))) - int(kNF4BinBase);
            code(j, x, uint32_t(k < 0 ? 0 : (k > kNF4RoundBins - 1 ? kNF4RoundBins - 1 : k)) << 4);
        }
    }
    packed = partial_wave(valid) ? p & nf4_nibble_mask(valid) : p;
    am = m;
}

// nf4_requant_round (the last step of a call) for a lane's 16 elements, a
// quarter of a block: the same arithmetic, the block maximum over 4 lanes.
// kExactRecip = false (fast mode): in the usual case r is v_rcp_f32's
// reciprocal (within 1 ulp of 1 / m) instead of the correctly rounded one, so
// x is within about 2 ulp of fl32(w * (1 / m)) and |x| <= 1 + 2^-22, which
// still takes bin 0 or 128 at the ends; a code can then differ from the
// exact quantizer's only where x lies within about 2^-23 of a midpoint.
template <bool kExactRecip>
__device__ __forceinline__ void nf4_requant_round16(const NF4Bin* bins, uint32_t valid, const float (&w)[16],
                                                    uint32_t (&packed)[2], float& am)
{
    float m = 0.0f;
#pragma unroll
    for (int j = 0; j < 16; ++j) m = fmaxf(m, fabsf(w[j]));
    m = max4(m);
    const bool usual = __float_as_uint(m) - kRecipLo <= kRecipHi - kRecipLo;
    const char* base = reinterpret_cast<const char*>(bins);
    // the codes of elements 8h .. 8h + 7 enter p[h] highest first (j = 15 .. 0)
    uint32_t p[2] = {0u, 0u};
    const auto code = [&](int j, float x, uint32_t off) {
        const float2 e = *reinterpret_cast<const float2*>(base + off);  // mid, lo
        const uint32_t c = __float_as_uint(e.y) + (x > e.x ? 1u : 0u);
        p[j >> 3] = (j & 7) == 7 ? c : shl4_or(p[j >> 3], c);
    };
    if (__builtin_amdgcn_ballot_w64(!usual) == 0) {  // uniform
        const float r = kExactRecip ? div_rn_normal(1.0f, m) : __builtin_amdgcn_rcpf(m);
#pragma unroll
        for (int j = 15; j >= 0; --j) {
            const float x = w[j] * r;
            const uint32_t t = __float_as_uint(__builtin_fmaf(x, 64.0f, kNF4BinMagic));
            code(j, x, (t << 4) - (kNF4BinBase << 4));  // 16 (t - base) = 16 b
        }
    } else {
        const float r = m > 0.0f ? 1.0f / m : 0.0f;
#pragma unroll
        for (int j = 15; j >= 0; --j) {
            const float x = w[j] * r;
            const float xs = x == x ? x : -2.0f;
            const int k = int(__float_as_uint(__builtin_fmaf(xs, 64.0f, kNF4BinMagic))) - int(kNF4BinBase);
            code(j, x, uint32_t(k < 0 ? 0 : (k > kNF4RoundBins - 1 ? kNF4RoundBins - 1 : k)) << 4);
        }
    }
    if (partial_wave16(valid)) {  // missing elements (a run of high bits of valid) get zero nibbles
        const uint32_t k = __builtin_popcount(valid);
        p[0] &= k >= 8 ? 0xFFFFFFFFu : (1u << (4 * k)) - 1u;
        p[1] &= k >= 16 ? 0xFFFFFFFFu : (k <= 8 ? 0u : (1u << (4 * (k - 8))) - 1u);
    }
    packed[0] = p[0];
    packed[1] = p[1];
    am = m;
}

}  // namespace mezo
