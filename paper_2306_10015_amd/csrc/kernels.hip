// kernels.hip — HIP kernels of the seeded perturbation engine (gfx950).
//
// One kernel applies any sequence of seeded perturbations to a whole parameter
// set in one pass: PerturbParameters (one record), the fused apply loop of one
// iteration (K records, the last flagged) and the late-joiner replay (T steps
// of records, each step's last flagged). Every element is read once and
// written once; its noise is regenerated in registers for every record.
//
// In place, or out of place from a source set of the same layout (theta =
// backup + sum c z: the restore of Algorithm 1 fused into the update).
//
// Launch shape: one launch per storage type, one workgroup per 4 KiB tile
// (1024 fp32 or 2048 bf16 elements); the workgroup finds its tensor with two scalar loads (tile -> tensor
// index -> descriptor). theta streams through with non-temporal 16-byte loads
// and stores (it is touched once per call, so it should not displace anything
// in the caches). Per lane, the seed-independent round-1 Philox product of each
// owned block is computed once and reused by every record; seed words, tensor
// id and coefficient are wave-uniform and live in SGPRs (scalar loads from the
// kernel arguments or from the staged record buffer).
#include <atomic>

#include "engine.hpp"
#include "launch.hpp"
#include "nf4.hpp"

namespace mezo {

template <bool kInline>
__device__ __forceinline__ const SeedRec& rec_at(const EngineArgs& a, uint32_t r)
{
    if constexpr (kInline)
        return a.inl[r];
    else
        return a.ext[r];
}

template <uint32_t kDtype>
struct Layout;
template <>
struct Layout<kF32> {
    static constexpr int kGroups = kGroupsF32;
    static constexpr uint64_t kPerGroup = 4;  // elements per 16-byte group
};
template <>
struct Layout<kBF16> {
    static constexpr int kGroups = kGroupsBF16;
    static constexpr uint64_t kPerGroup = 8;
};

// The 16-byte groups a lane owns in one tile, as loaded from memory. A group
// that runs past the end of its tensor is not loaded here (it stays zero) and
// is read element by element when the tile is processed.
template <int kGroups>
struct TileRaw {
    uint4 g[kGroups];
};

template <int kGroups>
__device__ __forceinline__ uint64_t group_index(uint64_t tile, int g)
{
    return tile * (kThreads * kGroups) + uint64_t(g) * kThreads + threadIdx.x;
}

// Parameter memory is global memory; saying so lets the compiler use global_*
// instead of flat_* instructions for addresses read from the tensor table.
#define MEZO_GLOBAL __attribute__((address_space(1)))
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef MEZO_GLOBAL u32x4_t gu32x4_t;
typedef MEZO_GLOBAL float gfloat_t;
typedef MEZO_GLOBAL uint16_t gu16_t;

__device__ __forceinline__ uint4 load_stream(uint64_t addr)
{
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const gu32x4_t*>(addr));
    return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ void store_stream(uint64_t addr, uint4 v)
{
    const u32x4_t w = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(w, reinterpret_cast<gu32x4_t*>(addr));
}

template <uint32_t kDtype>
__device__ __forceinline__ void load_tile(const TensorDesc& d, uint64_t src, uint64_t tile,
                                          TileRaw<Layout<kDtype>::kGroups>& raw)
{
    constexpr int kGroups = Layout<kDtype>::kGroups;
#pragma unroll
    for (int g = 0; g < kGroups; ++g) {
        const uint64_t grp = group_index<kGroups>(tile, g);
        if ((grp + 1) * Layout<kDtype>::kPerGroup <= d.numel)
            raw.g[g] = load_stream(src + grp * 16);
        else
            raw.g[g] = make_uint4(0u, 0u, 0u, 0u);
    }
}

// A tile that lies wholly inside its tensor (every tile but a tensor's last):
// no per-lane bounds, and each access is the tile's (uniform) base address
// plus a 32-bit lane offset.
template <uint32_t kDtype>
__device__ __forceinline__ void load_tile_full(uint64_t src, uint64_t tile, TileRaw<Layout<kDtype>::kGroups>& raw)
{
    constexpr int kGroups = Layout<kDtype>::kGroups;
    const gu32x4_t* base = reinterpret_cast<const gu32x4_t*>(src) + tile * (kThreads * kGroups);
#pragma unroll
    for (int g = 0; g < kGroups; ++g) {
        const u32x4_t v = __builtin_nontemporal_load(base + (uint32_t(g * kThreads) + threadIdx.x));
        raw.g[g] = make_uint4(v.x, v.y, v.z, v.w);
    }
}

// Cache-policy bits of a buffer store on gfx950: sc1 (16) | nt (2).
constexpr int kStorePolicy = 16 | 2;

template <int kGroups>
__device__ __forceinline__ void store_group_full(uint64_t dst, uint64_t tile, int g, uint4 v)
{
    // a buffer store over the tile's 4 KiB with the cache policy "sc1 nt"
    // (paired against "nt" alone: the 125M fp32 sweep 1.9% faster, the bf16
    // sweeps and the record loops unchanged)
    void* base = reinterpret_cast<void*>(dst + tile * (kThreads * kGroups * 16));
    const __amdgpu_buffer_rsrc_t r =
        __builtin_amdgcn_make_buffer_rsrc(base, (short)0, kThreads * kGroups * 16, 0x00020000);
    const u32x4_t w = {v.x, v.y, v.z, v.w};
    __builtin_amdgcn_raw_buffer_store_b128(w, r, (uint32_t(g * kThreads) + threadIdx.x) * 16u, 0, kStorePolicy);
}

// One tile of an fp32 tensor: each lane owns kGroups groups of 4 elements
// (one Philox block each).
template <bool kInline, bool kPortable>
__device__ __forceinline__ void tile_f32(const EngineArgs& a, const TensorDesc& d, uint64_t src,
                                         uint64_t tile, bool full, const TileRaw<kGroupsF32>& raw)
{
    constexpr int kGroups = kGroupsF32;
    const gfloat_t* in = reinterpret_cast<const gfloat_t*>(src);
    gfloat_t* out = reinterpret_cast<gfloat_t*>(d.data);
    const uint64_t numel = d.numel;
    float th[kGroups][4];
    float acc[kGroups][4];
    BlockPre pre[kGroups];
    uint64_t e0[kGroups];

#pragma unroll
    for (int g = 0; g < kGroups; ++g) {
        const uint64_t grp = group_index<kGroups>(tile, g);
        e0[g] = grp * 4;
        if (full || e0[g] + 4 <= numel) {
            th[g][0] = __uint_as_float(raw.g[g].x);
            th[g][1] = __uint_as_float(raw.g[g].y);
            th[g][2] = __uint_as_float(raw.g[g].z);
            th[g][3] = __uint_as_float(raw.g[g].w);
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) th[g][j] = (e0[g] + j < numel) ? in[e0[g] + j] : 0.0f;
        }
        pre[g] = block_pre(uint32_t((d.first >> 2) + grp));  // block of the logical tensor
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[g][j] = 0.0f;
    }

    const auto accumulate = [&](uint32_t r) {
        const SeedRec& rec = rec_at<kInline>(a, r);
        const SeedUniform u = seed_uniform(rec, d.tensor_id);
        const float c = rec.coef;
#pragma unroll
        for (int g = 0; g < kGroups; ++g) {
            uint32_t w0, w1, w2, w3;
            philox_words(u, pre[g], w0, w1, w2, w3);
            accumulate4<kPortable>(c, w0, w1, w2, w3, acc[g][0], acc[g][1], acc[g][2], acc[g][3]);
        }
    };
    // the last record ends the call's last step: peeled off the loop, it
    // needs no reset of acc afterwards
    for (uint32_t r = 0; r + 1 < a.n_rec; ++r) {
        accumulate(r);
        if (rec_at<kInline>(a, r).last) {
#pragma unroll
            for (int g = 0; g < kGroups; ++g)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    th[g][j] = th[g][j] + acc[g][j];
                    acc[g][j] = 0.0f;
                }
        }
    }
    if (a.n_rec > 0) {
        accumulate(a.n_rec - 1);
#pragma unroll
        for (int g = 0; g < kGroups; ++g)
#pragma unroll
            for (int j = 0; j < 4; ++j) th[g][j] = th[g][j] + acc[g][j];
    }

    if (full) {
#pragma unroll
        for (int g = 0; g < kGroups; ++g)
            store_group_full<kGroups>(d.data, tile, g,
                                      make_uint4(__float_as_uint(th[g][0]), __float_as_uint(th[g][1]),
                                                 __float_as_uint(th[g][2]), __float_as_uint(th[g][3])));
        return;
    }
#pragma unroll
    for (int g = 0; g < kGroups; ++g) {
        if (e0[g] + 4 <= numel) {
            store_stream(d.data + e0[g] * 4, make_uint4(__float_as_uint(th[g][0]), __float_as_uint(th[g][1]),
                                                        __float_as_uint(th[g][2]), __float_as_uint(th[g][3])));
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (e0[g] + j < numel) out[e0[g] + j] = th[g][j];
        }
    }
}

// A lane's bf16 groups of 8 elements (two Philox blocks each) through all
// records. theta stays packed: after every step it is a bf16 value again, so
// the packed pairs lose nothing; a step ends with one RNE rounding of
// theta + acc.
template <bool kInline, bool kPortable>
__device__ __forceinline__ void groups_bf16(const EngineArgs& a, const TensorDesc& d, uint64_t tile,
                                            uint32_t (&th)[kGroupsBF16][4])
{
    constexpr int kGroups = kGroupsBF16;
    float acc[kGroups][8];
    BlockPre pre[kGroups][2];
#pragma unroll
    for (int g = 0; g < kGroups; ++g) {
        const uint64_t grp = group_index<kGroups>(tile, g);
        const uint64_t blk = (d.first >> 2) + 2 * grp;  // block of the logical tensor
        pre[g][0] = block_pre(uint32_t(blk));
        pre[g][1] = block_pre(uint32_t(blk + 1));
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[g][j] = 0.0f;
    }
    const auto accumulate = [&](uint32_t r) {
        const SeedRec& rec = rec_at<kInline>(a, r);
        const SeedUniform u = seed_uniform(rec, d.tensor_id);
        const float c = rec.coef;
#pragma unroll
        for (int g = 0; g < kGroups; ++g)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                uint32_t w0, w1, w2, w3;
                philox_words(u, pre[g][h], w0, w1, w2, w3);
                accumulate4<kPortable>(c, w0, w1, w2, w3, acc[g][4 * h + 0], acc[g][4 * h + 1],
                                       acc[g][4 * h + 2], acc[g][4 * h + 3]);
            }
    };
    const auto step_end = [&]() {
#pragma unroll
        for (int g = 0; g < kGroups; ++g)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                th[g][j] = pack_bf16(bf16_lo(th[g][j]) + acc[g][2 * j], bf16_hi(th[g][j]) + acc[g][2 * j + 1]);
    };
    // the last record ends the call's last step: peeled off the loop, it
    // needs no reset of acc afterwards
    for (uint32_t r = 0; r + 1 < a.n_rec; ++r) {
        accumulate(r);
        if (rec_at<kInline>(a, r).last) {
            step_end();
#pragma unroll
            for (int g = 0; g < kGroups; ++g)
#pragma unroll
                for (int j = 0; j < 8; ++j) acc[g][j] = 0.0f;
        }
    }
    if (a.n_rec > 0) {
        accumulate(a.n_rec - 1);
        step_end();
    }
}

// One tile of a bf16 tensor: each lane owns kGroupsBF16 groups of 8 elements.
template <bool kInline, bool kPortable>
__device__ __forceinline__ void tile_bf16(const EngineArgs& a, const TensorDesc& d, uint64_t src,
                                          uint64_t tile, bool full, const TileRaw<kGroupsBF16>& raw)
{
    constexpr int kGroups = kGroupsBF16;
    const gu16_t* in = reinterpret_cast<const gu16_t*>(src);
    gu16_t* out = reinterpret_cast<gu16_t*>(d.data);
    const uint64_t numel = d.numel;
    uint32_t th[kGroups][4];
    uint64_t e0[kGroups];
#pragma unroll
    for (int g = 0; g < kGroups; ++g) {
        e0[g] = group_index<kGroups>(tile, g) * 8;
        if (full || e0[g] + 8 <= numel) {
            th[g][0] = raw.g[g].x;
            th[g][1] = raw.g[g].y;
            th[g][2] = raw.g[g].z;
            th[g][3] = raw.g[g].w;
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const uint32_t lo = (e0[g] + 2 * j < numel) ? uint32_t(in[e0[g] + 2 * j]) : 0u;
                const uint32_t hi = (e0[g] + 2 * j + 1 < numel) ? uint32_t(in[e0[g] + 2 * j + 1]) : 0u;
                th[g][j] = lo | (hi << 16);
            }
        }
    }
    groups_bf16<kInline, kPortable>(a, d, tile, th);
    if (full) {
#pragma unroll
        for (int g = 0; g < kGroups; ++g)
            store_group_full<kGroups>(d.data, tile, g, make_uint4(th[g][0], th[g][1], th[g][2], th[g][3]));
        return;
    }
#pragma unroll
    for (int g = 0; g < kGroups; ++g) {
        if (e0[g] + 8 <= numel) {
            store_stream(d.data + e0[g] * 2, make_uint4(th[g][0], th[g][1], th[g][2], th[g][3]));
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (e0[g] + j < numel) out[e0[g] + j] = uint16_t(th[g][j >> 1] >> (16 * (j & 1)));
        }
    }
}

// ---- NF4 storage (the 4-bit forward-only variant) -----------------------------
// A lane owns 8 consecutive elements (one dword of codes); the 8 lanes
// tid & ~7 .. tid | 7 own one 64-element block and share its absmax. Codes
// become values through a 16-entry table and values become codes through the
// 128-bin table of nf4.hpp, both copied into LDS by every workgroup.

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

// kFull: a tile wholly inside its tensor, where every lane's 8 elements exist
// (no masks, no bounds).
template <bool kInline, bool kPortable, bool kFull>
__device__ __forceinline__ void tile_nf4(const EngineArgs& a, const TensorDesc& d, uint64_t e0, uint32_t packed,
                                         float am, const NF4Lds& s)
{
    const uint32_t valid = kFull ? 0xFFu : nf4_valid(e0, d.numel);
    float w[8];
    nf4_dequant(s, packed, am, valid, w);
    float acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = 0.0f;
    const uint64_t blk = (d.first + e0) >> 2;  // block of the logical tensor
    const BlockPre pre0 = block_pre(uint32_t(blk));
    const BlockPre pre1 = block_pre(uint32_t(blk + 1));
    const auto accumulate = [&](uint32_t r) {
        const SeedRec& rec = rec_at<kInline>(a, r);
        const SeedUniform u = seed_uniform(rec, d.tensor_id);
        const float c = rec.coef;
        uint32_t w0, w1, w2, w3;
        philox_words(u, pre0, w0, w1, w2, w3);
        accumulate4<kPortable>(c, w0, w1, w2, w3, acc[0], acc[1], acc[2], acc[3]);
        philox_words(u, pre1, w0, w1, w2, w3);
        accumulate4<kPortable>(c, w0, w1, w2, w3, acc[4], acc[5], acc[6], acc[7]);
    };
    const auto step_end = [&]() {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            w[j] = w[j] + acc[j];
            acc[j] = 0.0f;
        }
        if (partial_wave(valid)) {  // only waves that reach a tensor's end
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (!((valid >> j) & 1u)) w[j] = 0.0f;
        }
    };
    if (a.n_rec == 0) {  // out of place with nothing to apply: a copy
        nf4_store<kFull>(d.data, d.aux, e0, d.numel, packed, am);
        return;
    }
    // every record list ends a step with its last record, which is peeled off
    // the loop: its quantization needs no values for a next step
    for (uint32_t r = 0; r + 1 < a.n_rec; ++r) {
        accumulate(r);
        if (rec_at<kInline>(a, r).last) {
            step_end();
            nf4_requant<true>(s.bin, valid, w, packed, am);
        }
    }
    accumulate(a.n_rec - 1);
    step_end();
    nf4_requant<false>(s.bin, valid, w, packed, am);
    nf4_store<kFull>(d.data, d.aux, e0, d.numel, packed, am);
}

// kShort (NF4 only): a call of at most two records, where the per-tile work
// outweighs the record loop; whole tiles then take a copy of the path compiled
// without bounds or masks. Long record lists keep a single copy of the loop
// (a second one costs the loop more than the tiles gain).
template <bool kInline, uint32_t kDtype, bool kPortable, bool kShort = false>
__global__ __launch_bounds__(kThreads) void engine_kernel(EngineArgs a)
{
    const uint64_t tile = blockIdx.x;  // the grid is exactly the tiles of this table
    const uint32_t ti = a.tile_tensor[tile];
    const TensorDesc d = a.tensors[ti];
    if constexpr (kDtype == kNF4) {
        __shared__ NF4Lds lds;
        // out of place: read tensor ti of the source set (same layout), write d
        const uint64_t codes = a.src_tensors ? a.src_tensors[ti].data : d.data;
        const uint64_t absmax = a.src_tensors ? a.src_tensors[ti].aux : d.aux;
        const uint64_t local = tile - d.tile_begin;
        const uint64_t e0 = local * kTileNF4 + threadIdx.x * 8u;
        uint32_t packed;
        float am;
        if (kShort && (local + 1) * kTileNF4 <= d.numel) {  // uniform: all but a tensor's last tile
            nf4_load<true>(codes, absmax, e0, d.numel, packed, am);
            nf4_lds_init(lds);
            tile_nf4<kInline, kPortable, true>(a, d, e0, packed, am, lds);
        } else {
            nf4_load(codes, absmax, e0, d.numel, packed, am);
            nf4_lds_init(lds);
            tile_nf4<kInline, kPortable, false>(a, d, e0, packed, am, lds);
        }
    } else {
        // out of place: read tensor ti of the source set (same layout), write d
        const uint64_t src = a.src_tensors ? a.src_tensors[ti].data : d.data;
        const uint64_t local = tile - d.tile_begin;
        constexpr uint64_t kTileElems = kThreads * Layout<kDtype>::kGroups * Layout<kDtype>::kPerGroup;
        const bool full = (local + 1) * kTileElems <= d.numel;  // uniform: all but a tensor's last tile
        TileRaw<Layout<kDtype>::kGroups> raw;
        if (full)
            load_tile_full<kDtype>(src, local, raw);
        else
            load_tile<kDtype>(d, src, local, raw);
        if constexpr (kDtype == kF32)
            tile_f32<kInline, kPortable>(a, d, src, local, full, raw);
        else
            tile_bf16<kInline, kPortable>(a, d, src, local, full, raw);
    }
}

// One lane's 8 elements of nf4_quantize_kernel; kFull: they all exist.
template <bool kFull>
__device__ __forceinline__ void nf4_quantize_tile(const NF4ConvArgs& a, const NF4Bin* bins, uint64_t e0)
{
    const uint32_t valid = kFull ? 0xFFu : nf4_valid(e0, a.n);
    float w[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) w[j] = 0.0f;
    if (a.dtype == kF32) {
        const gfloat_t* in = reinterpret_cast<const gfloat_t*>(a.values);
        if (kFull || valid == 0xFFu) {
            const uint4 v0 = load_stream(a.values + e0 * 4);
            const uint4 v1 = load_stream(a.values + e0 * 4 + 16);
            const uint32_t u[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
#pragma unroll
            for (int j = 0; j < 8; ++j) w[j] = __uint_as_float(u[j]);
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if ((valid >> j) & 1u) w[j] = in[e0 + j];
        }
    } else {
        const gu16_t* in = reinterpret_cast<const gu16_t*>(a.values);
        if (kFull || valid == 0xFFu) {
            const uint4 v = load_stream(a.values + e0 * 2);
            const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                w[2 * j] = bf16_lo(u[j]);
                w[2 * j + 1] = bf16_hi(u[j]);
            }
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if ((valid >> j) & 1u) w[j] = __uint_as_float(uint32_t(in[e0 + j]) << 16);
        }
    }
    uint32_t packed;
    float am;
    nf4_requant<false>(bins, valid, w, packed, am);
    nf4_store<kFull>(a.codes, a.absmax, e0, a.n, packed, am);
}

// Standalone NF4 conversions (one tile of 2048 elements per workgroup).
__global__ __launch_bounds__(kThreads) void nf4_quantize_kernel(NF4ConvArgs a)
{
    // one copy of the bin table per wave: a wave fills its own and reads it
    // after its writes (one wave's LDS accesses complete in order), so the
    // waves of a workgroup never wait for each other
    __shared__ NF4Bin wave_bins[kThreads / 64][kNF4Bins];
    NF4Bin* bins = wave_bins[threadIdx.x >> 6];
    const uint32_t lane = threadIdx.x & 63u;
    bins[lane] = kNF4Table.bin[lane];
    bins[lane + 64] = kNF4Table.bin[lane + 64];
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const uint64_t e0 = uint64_t(blockIdx.x) * kTileNF4 + threadIdx.x * 8u;
    if ((uint64_t(blockIdx.x) + 1) * kTileNF4 <= a.n)  // uniform: every tile but the last
        nf4_quantize_tile<true>(a, bins, e0);
    else
        nf4_quantize_tile<false>(a, bins, e0);
}

// The 16 values held by lanes 0..15 of every wave (lane l: value l mod 16).
__device__ __forceinline__ uint32_t nf4_value_lanes()
{
    return __float_as_uint(kNF4Values[threadIdx.x & 15u]);
}

// nf4_dequant with the value of each code fetched from the lane that holds it
// (a lane permute: no LDS table to fill, no workgroup barrier).
__device__ __forceinline__ void nf4_dequant_lanes(uint32_t table, uint32_t packed, float am, uint32_t valid,
                                                  float (&w)[8])
{
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int addr = int(((packed >> (4 * j)) & 15u) << 2);  // byte address of the code's lane
        w[j] = __uint_as_float(uint32_t(__builtin_amdgcn_ds_bpermute(addr, int(table)))) * am;
    }
    if (valid != 0xFFu) {  // a tensor's last lanes only
#pragma unroll
        for (int j = 0; j < 8; ++j)
            if (!((valid >> j) & 1u)) w[j] = 0.0f;
    }
}

// One lane's 8 elements of nf4_dequantize_kernel; kFull: they all exist.
template <bool kFull>
__device__ __forceinline__ void nf4_dequantize_tile(const NF4ConvArgs& a, uint64_t e0)
{
    const uint32_t valid = kFull ? 0xFFu : nf4_valid(e0, a.n);
    const uint32_t table = nf4_value_lanes();
    uint32_t packed;
    float am;
    nf4_load<kFull>(a.codes, a.absmax, e0, a.n, packed, am);
    float w[8];
    nf4_dequant_lanes(table, packed, am, valid, w);
    if (a.dtype == kF32) {
        gfloat_t* out = reinterpret_cast<gfloat_t*>(a.values);
        if constexpr (kFull) {
            // the workgroup's 8 KiB of output through a buffer resource, with
            // the engine's store policy
            const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
                reinterpret_cast<void*>(a.values + uint64_t(blockIdx.x) * kTileNF4 * 4), (short)0,
                int(kTileNF4 * 4), 0x00020000);
            const u32x4_t lo = {__float_as_uint(w[0]), __float_as_uint(w[1]), __float_as_uint(w[2]),
                                __float_as_uint(w[3])};
            const u32x4_t hi = {__float_as_uint(w[4]), __float_as_uint(w[5]), __float_as_uint(w[6]),
                                __float_as_uint(w[7])};
            __builtin_amdgcn_raw_buffer_store_b128(lo, r, threadIdx.x * 32u, 0, kStorePolicy);
            __builtin_amdgcn_raw_buffer_store_b128(hi, r, threadIdx.x * 32u + 16u, 0, kStorePolicy);
        } else if (valid == 0xFFu) {
            store_stream(a.values + e0 * 4, make_uint4(__float_as_uint(w[0]), __float_as_uint(w[1]),
                                                       __float_as_uint(w[2]), __float_as_uint(w[3])));
            store_stream(a.values + e0 * 4 + 16, make_uint4(__float_as_uint(w[4]), __float_as_uint(w[5]),
                                                            __float_as_uint(w[6]), __float_as_uint(w[7])));
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if ((valid >> j) & 1u) out[e0 + j] = w[j];
        }
    } else {
        gu16_t* out = reinterpret_cast<gu16_t*>(a.values);
        if constexpr (kFull) {
            const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
                reinterpret_cast<void*>(a.values + uint64_t(blockIdx.x) * kTileNF4 * 2), (short)0,
                int(kTileNF4 * 2), 0x00020000);
            const u32x4_t v = {pack_bf16(w[0], w[1]), pack_bf16(w[2], w[3]), pack_bf16(w[4], w[5]),
                               pack_bf16(w[6], w[7])};
            __builtin_amdgcn_raw_buffer_store_b128(v, r, threadIdx.x * 16u, 0, kStorePolicy);
        } else if (valid == 0xFFu) {
            store_stream(a.values + e0 * 2, make_uint4(pack_bf16(w[0], w[1]), pack_bf16(w[2], w[3]),
                                                       pack_bf16(w[4], w[5]), pack_bf16(w[6], w[7])));
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if ((valid >> j) & 1u) out[e0 + j] = to_bf16(w[j]);
        }
    }
}

__global__ __launch_bounds__(kThreads) void nf4_dequantize_kernel(NF4ConvArgs a)
{
    const uint64_t e0 = uint64_t(blockIdx.x) * kTileNF4 + threadIdx.x * 8u;
    if ((uint64_t(blockIdx.x) + 1) * kTileNF4 <= a.n)  // uniform: every tile but the last
        nf4_dequantize_tile<true>(a, e0);
    else
        nf4_dequantize_tile<false>(a, e0);
}

// Inspection: RNG words and Gaussians of a range of elements, one Philox
// block per lane, through the same generator functions as the engine.
__global__ __launch_bounds__(kThreads) void generate_kernel(GenArgs a)
{
    const uint64_t blk = (a.first >> 2) + uint64_t(blockIdx.x) * kThreads + threadIdx.x;
    const uint64_t end = a.first + a.count;
    const uint64_t eb = blk * 4;
    if (eb >= end) return;
    const SeedUniform u = seed_uniform(a.rec, a.tensor_id);
    uint32_t w[4];
    philox_words(u, block_pre(uint32_t(blk)), w[0], w[1], w[2], w[3]);
    const Z4 z4 = a.portable ? gauss4_portable(w[0], w[1], w[2], w[3]) : gauss4(w[0], w[1], w[2], w[3]);
    const float z[4] = {z4.z0, z4.z1, z4.z2, z4.z3};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const uint64_t e = eb + j;
        if (e < a.first || e >= end) continue;
        const uint64_t i = e - a.first;
        if (a.words) a.words[i] = w[j];
        if (a.z) a.z[i] = z[j];
    }
}

// ---- checksum of theta (ChecksumMatch, Algorithm 1) ---------------------------
// Read-only stream over the same tiles as the engine; every lane sums the
// mixes of its 8-byte chunks, a workgroup reduces across lanes and waves and
// adds its sum to the output with one 64-bit atomic. Sums mod 2^64 commute, so
// the grid shape and the order of the atomics do not change the result.

__device__ __forceinline__ uint64_t fmix64(uint64_t x)
{
    x ^= x >> 33;
    x *= kFmixA;
    x ^= x >> 33;
    x *= kFmixB;
    x ^= x >> 33;
    return x;
}

// Reduce every lane's sum across the workgroup and add it to *out with one
// 64-bit atomic (all lanes of the workgroup must call it).
__device__ __forceinline__ void add_workgroup_sum(uint64_t sum, unsigned long long* out)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) sum += __shfl_xor(sum, off);
    __shared__ uint64_t part[kThreads / 64];
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = sum;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint64_t s = 0;
#pragma unroll
        for (int i = 0; i < kThreads / 64; ++i) s += part[i];
        atomicAdd(out, static_cast<unsigned long long>(s));
    }
}

// One lane's share of a tile that lies wholly inside its tensor (every tile
// but a tensor's last): no bounds, the tile's scalar base plus a 32-bit lane
// offset, and chunk numbers as a uniform part plus the lane's constant one.
template <int kGroups>
__device__ __forceinline__ uint64_t checksum_full_tile(uint64_t data, uint64_t local, uint64_t cpos_tile,
                                                       uint64_t tmix, const uint64_t (&cpos_lane)[kGroups])
{
    const gu32x4_t* base = reinterpret_cast<const gu32x4_t*>(data) + local * (kThreads * kGroups);
    uint64_t sum = 0;
#pragma unroll
    for (int g = 0; g < kGroups; ++g) {
        const u32x4_t v = __builtin_nontemporal_load(base + (uint32_t(g * kThreads) + threadIdx.x));
        const uint64_t p0 = cpos_tile + cpos_lane[g];  // (its first chunk's number) * kChunkPos
        const uint64_t lo = uint64_t(v.x) | (uint64_t(v.y) << 32);
        const uint64_t hi = uint64_t(v.z) | (uint64_t(v.w) << 32);
        sum += fmix64(lo ^ p0 ^ tmix);
        sum += fmix64(hi ^ (p0 + kChunkPos) ^ tmix);
    }
    return sum;
}

template <uint32_t kDtype>
__global__ __launch_bounds__(kThreads) void checksum_kernel(ChecksumArgs a)
{
    constexpr int kGroups = Layout<kDtype>::kGroups;
    constexpr uint64_t kPer = Layout<kDtype>::kPerGroup;
    constexpr uint64_t kEsz = 16 / kPer;
    constexpr uint64_t kTileElems = uint64_t(kThreads) * kGroups * kPer;
    // chunk number of a lane's group g within its tile, times kChunkPos
    uint64_t cpos_lane[kGroups];
#pragma unroll
    for (int g = 0; g < kGroups; ++g) {
        cpos_lane[g] = 2 * (uint64_t(g) * kThreads + threadIdx.x) * kChunkPos;
        // opaque from here on: otherwise the compiler folds uniform + lane
        // constant back into one per-lane 64-bit multiply in every tile
        asm("" : "+v"(cpos_lane[g]));
    }
    uint64_t sum = 0;
    for (uint64_t tile = blockIdx.x; tile < a.total_tiles; tile += gridDim.x) {
        const TensorDesc d = a.tensors[a.tile_tensor[tile]];
        const uint64_t local = tile - d.tile_begin;
        const uint64_t nbytes = d.numel * kEsz;
        const uint64_t nchunks = (nbytes + 7) / 8;
        const uint64_t cbase = d.first * kEsz / 8;  // chunk number of the shard's first byte
        const uint64_t tmix = uint64_t(d.tensor_id) * kChunkTensor;
        if ((local + 1) * kTileElems <= d.numel) {  // uniform
            const uint64_t cpos_tile = (cbase + 2 * local * (kThreads * kGroups)) * kChunkPos;
            sum += checksum_full_tile<kGroups>(d.data, local, cpos_tile, tmix, cpos_lane);
            continue;
        }
#pragma unroll
        for (int g = 0; g < kGroups; ++g) {
            const uint64_t grp = group_index<kGroups>(local, g);
            const uint64_t c0 = grp * 2;  // the group's first chunk within the shard
            if (c0 >= nchunks) continue;
            uint4 v;
            if ((grp + 1) * kPer <= d.numel) {
                v = load_stream(d.data + grp * 16);
            } else {
                // tail: read the elements that exist, zero the rest
                uint32_t w[4] = {0u, 0u, 0u, 0u};
                if constexpr (kDtype == kF32) {
                    const MEZO_GLOBAL uint32_t* in = reinterpret_cast<const MEZO_GLOBAL uint32_t*>(d.data);
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        if (grp * 4 + j < d.numel) w[j] = in[grp * 4 + j];
                } else {
                    const gu16_t* in = reinterpret_cast<const gu16_t*>(d.data);
#pragma unroll
                    for (int j = 0; j < 8; ++j)
                        if (grp * 8 + j < d.numel) w[j >> 1] |= uint32_t(in[grp * 8 + j]) << (16 * (j & 1));
                }
                v = make_uint4(w[0], w[1], w[2], w[3]);
            }
            const uint64_t lo = uint64_t(v.x) | (uint64_t(v.y) << 32);
            const uint64_t hi = uint64_t(v.z) | (uint64_t(v.w) << 32);
            sum += fmix64(lo ^ ((cbase + c0) * kChunkPos) ^ tmix);
            if (c0 + 1 < nchunks) sum += fmix64(hi ^ ((cbase + c0 + 1) * kChunkPos) ^ tmix);
        }
    }
    add_workgroup_sum(sum, a.out);
}

// NF4 tensors: the code bytes zero-padded to whole chunks, then the absmax
// values, chunk numbers continuing. One wave per tile of 2048 elements: every
// lane reads 16 code bytes (two chunks) and lanes 0..7 also 16 bytes of the
// tile's 128 absmax bytes.
__global__ __launch_bounds__(kThreads) void checksum_nf4_kernel(ChecksumArgs a)
{
    constexpr uint32_t kWaves = kThreads / 64;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint32_t lane = threadIdx.x & 63u;
    // position terms of a lane's chunks within a tile, computed once (opaque
    // to the compiler, as in checksum_kernel): code chunks 2 lane, 2 lane + 1;
    // absmax chunk lane (lanes 0..15)
    uint64_t cpos_code = 2 * uint64_t(lane) * kChunkPos;
    uint64_t cpos_abs = uint64_t(lane & 15u) * kChunkPos;
    asm("" : "+v"(cpos_code));
    asm("" : "+v"(cpos_abs));
    uint64_t sum = 0;
    for (uint64_t tile = uint64_t(blockIdx.x) * kWaves + wave; tile < a.total_tiles;
         tile += uint64_t(gridDim.x) * kWaves) {
        const TensorDesc d = a.tensors[a.tile_tensor[tile]];
        const uint64_t local = tile - d.tile_begin;
        const uint64_t cbytes = (d.numel + 1) / 2;
        const uint64_t cchunks = (cbytes + 7) / 8;
        const uint64_t abytes = 4 * ((d.numel + kNF4Block - 1) / kNF4Block);
        const uint64_t tmix = uint64_t(d.tensor_id) * kChunkTensor;
        if ((local + 1) * kTileNF4 <= d.numel) {  // uniform: a whole tile, 32 whole blocks
            const gu32x4_t* codes = reinterpret_cast<const gu32x4_t*>(d.data) + local * 64;
            const u32x4_t v = __builtin_nontemporal_load(codes + lane);
            // the tile's 128 absmax bytes as 16 chunks on lanes 0..15; every
            // lane loads (lane mod 16), so that both loads issue before any mix
            const MEZO_GLOBAL uint64_t* am = reinterpret_cast<const MEZO_GLOBAL uint64_t*>(d.aux) + local * 16;
            const uint64_t f = __builtin_nontemporal_load(am + (lane & 15u));
            const uint64_t p0 = 128 * local * kChunkPos + cpos_code;
            sum += fmix64((uint64_t(v.x) | (uint64_t(v.y) << 32)) ^ p0 ^ tmix);
            sum += fmix64((uint64_t(v.z) | (uint64_t(v.w) << 32)) ^ (p0 + kChunkPos) ^ tmix);
            const uint64_t fm = fmix64(f ^ ((cchunks + 16 * local) * kChunkPos + cpos_abs) ^ tmix);
            sum += lane < 16u ? fm : 0u;
            continue;
        }
        // codes: bytes [16u, 16u + 16) = chunks 2u, 2u + 1
        const uint64_t u = local * 64 + lane;
        if (16 * u < cbytes) {
            uint64_t lo = 0, hi = 0;
            if (16 * u + 16 <= cbytes) {
                const uint4 v = load_stream(d.data + 16 * u);
                lo = uint64_t(v.x) | (uint64_t(v.y) << 32);
                hi = uint64_t(v.z) | (uint64_t(v.w) << 32);
            } else {
                const MEZO_GLOBAL uint8_t* b = reinterpret_cast<const MEZO_GLOBAL uint8_t*>(d.data);
                for (uint64_t k = 16 * u; k < cbytes; ++k) {
                    const uint64_t byte = uint64_t(b[k]);
                    const uint64_t off = k - 16 * u;
                    if (off < 8)
                        lo |= byte << (8 * off);
                    else
                        hi |= byte << (8 * (off - 8));
                }
            }
            sum += fmix64(lo ^ (2 * u * kChunkPos) ^ tmix);
            if (16 * u + 8 < cbytes) sum += fmix64(hi ^ ((2 * u + 1) * kChunkPos) ^ tmix);
        }
        // absmax: bytes [ab, ab + 16) = absmax chunks k0, k0 + 1
        const uint64_t ab = local * (kTileNF4 / kNF4Block * 4) + 16 * uint64_t(lane);
        if (lane < kTileNF4 / kNF4Block * 4 / 16 && ab < abytes) {
            const uint64_t k0 = ab / 8;
            uint32_t f[4] = {0u, 0u, 0u, 0u};
            if (ab + 16 <= abytes) {
                const uint4 v = load_stream(d.aux + ab);
                f[0] = v.x;
                f[1] = v.y;
                f[2] = v.z;
                f[3] = v.w;
            } else {
                const MEZO_GLOBAL uint32_t* am = reinterpret_cast<const MEZO_GLOBAL uint32_t*>(d.aux);
                for (uint64_t k = ab; k < abytes; k += 4) f[(k - ab) / 4] = am[k / 4];
            }
            sum += fmix64((uint64_t(f[0]) | (uint64_t(f[1]) << 32)) ^ ((cchunks + k0) * kChunkPos) ^ tmix);
            if (ab + 8 < abytes)
                sum += fmix64((uint64_t(f[2]) | (uint64_t(f[3]) << 32)) ^ ((cchunks + k0 + 1) * kChunkPos) ^ tmix);
        }
    }
    add_workgroup_sum(sum, a.out);
}

__global__ void zero_u64_kernel(unsigned long long* out)
{
    if (threadIdx.x == 0 && blockIdx.x == 0) *out = 0ull;
}

// ---- host-side launchers ----------------------------------------------------

namespace {
// Launch a one-argument kernel and return the status of this launch itself
// (not the thread's last HIP error, which may hold an earlier failure of
// another caller's call).
template <class Arg>
hipError_t launch1(void (*kernel)(Arg), dim3 g, dim3 b, hipStream_t stream, Arg arg)
{
    void* params[] = {&arg};
    return hipLaunchKernel(reinterpret_cast<const void*>(kernel), g, b, params, 0, stream);
}

template <bool kInline, bool kPortable>
hipError_t launch_dtype(const EngineArgs& args, uint32_t dtype, dim3 g, dim3 b, hipStream_t stream)
{
    if (dtype == kF32) return launch1(engine_kernel<kInline, kF32, kPortable>, g, b, stream, args);
    if (dtype == kBF16) return launch1(engine_kernel<kInline, kBF16, kPortable>, g, b, stream, args);
    if constexpr (kInline) {
        if (args.n_rec <= 2) return launch1(engine_kernel<kInline, kNF4, kPortable, true>, g, b, stream, args);
    }
    return launch1(engine_kernel<kInline, kNF4, kPortable>, g, b, stream, args);
}
}  // namespace

hipError_t launch_engine(const EngineArgs& args, uint32_t dtype, bool portable, hipStream_t stream)
{
    if (args.total_tiles == 0) return hipSuccess;
    if (args.total_tiles > uint64_t(0x7FFFFFFF) || dtype >= kStorageTypes) return hipErrorInvalidValue;
    const bool inl = args.n_rec <= kInlineRecs;
    const dim3 g{uint32_t(args.total_tiles)};
    const dim3 b{uint32_t(kThreads)};
    if (inl)
        return portable ? launch_dtype<true, true>(args, dtype, g, b, stream)
                        : launch_dtype<true, false>(args, dtype, g, b, stream);
    return portable ? launch_dtype<false, true>(args, dtype, g, b, stream)
                    : launch_dtype<false, false>(args, dtype, g, b, stream);
}

hipError_t launch_generate(const GenArgs& args, hipStream_t stream)
{
    // At most 2^26 blocks (2^28 elements) per launch keeps the grid small.
    const uint64_t kChunk = uint64_t(1) << 28;
    GenArgs a = args;
    uint64_t left = args.count;
    uint64_t first = args.first;
    uint64_t done = 0;
    while (left > 0) {
        const uint64_t n = left < kChunk ? left : kChunk;
        a.first = first;
        a.count = n;
        a.words = args.words ? args.words + done : nullptr;
        a.z = args.z ? args.z + done : nullptr;
        const uint64_t nblk = ((first + n - 1) >> 2) - (first >> 2) + 1;
        const uint64_t grid = (nblk + kThreads - 1) / kThreads;
        const hipError_t e = launch1(generate_kernel, dim3(uint32_t(grid)), dim3(kThreads), stream, a);
        if (e != hipSuccess) return e;
        left -= n;
        first += n;
        done += n;
    }
    return hipSuccess;
}

namespace {
constexpr int kMaxDevices = 64;
std::atomic<int> g_cus[kMaxDevices];  // compute units per device, 0 = not yet asked
}  // namespace

hipError_t launch_checksum(const ChecksumArgs* tables, const uint32_t* dtypes, int n_tables,
                           unsigned long long* out, int device, hipStream_t stream)
{
    if (device < 0 || device >= kMaxDevices) return hipErrorInvalidValue;
    int cus = g_cus[device].load(std::memory_order_relaxed);
    if (cus == 0) {
        hipError_t e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device);
        if (e != hipSuccess) return e;
        g_cus[device].store(cus, std::memory_order_relaxed);
    }
    hipError_t e = launch1(zero_u64_kernel, dim3(1), dim3(64), stream, out);
    if (e != hipSuccess) return e;
    for (int i = 0; i < n_tables; ++i) {
        if (tables[i].total_tiles == 0) continue;
        // as many workgroups as fill the device (8 per CU), each striding over
        // tiles (NF4: four tiles at a time, one per wave)
        const uint64_t per_wg = dtypes[i] == kNF4 ? kThreads / 64 : 1;
        const uint64_t need = (tables[i].total_tiles + per_wg - 1) / per_wg;
        const uint64_t cap = uint64_t(cus) * 8;
        const uint64_t grid = need < cap ? need : cap;
        const dim3 g{uint32_t(grid)};
        const dim3 b{uint32_t(kThreads)};
        if (dtypes[i] == kF32)
            e = launch1(checksum_kernel<kF32>, g, b, stream, tables[i]);
        else if (dtypes[i] == kBF16)
            e = launch1(checksum_kernel<kBF16>, g, b, stream, tables[i]);
        else
            e = launch1(checksum_nf4_kernel, g, b, stream, tables[i]);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_nf4(const NF4ConvArgs& args, bool quantize, hipStream_t stream)
{
    const uint64_t tiles = (args.n + kTileNF4 - 1) / kTileNF4;
    if (tiles == 0) return hipSuccess;
    if (tiles > uint64_t(0x7FFFFFFF)) return hipErrorInvalidValue;
    const dim3 g{uint32_t(tiles)};
    const dim3 b{uint32_t(kThreads)};
    return launch1(quantize ? nf4_quantize_kernel : nf4_dequantize_kernel, g, b, stream, args);
}

}  // namespace mezo
