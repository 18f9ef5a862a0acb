// engine_dense.hip — the engine kernel on fp32 and bf16 storage (gfx950).
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
// (1024 fp32 or 2048 bf16 elements); the workgroup finds its tensor with two
// scalar loads (tile -> tensor index -> descriptor). theta streams through
// with non-temporal 16-byte loads and stores (it is touched once per call, so
// it should not displace anything in the caches). Per lane, the
// seed-independent round-1 Philox product of each owned block is computed once
// and reused by every record; seed words, tensor id and coefficient are
// wave-uniform and live in SGPRs (scalar loads from the kernel arguments or
// from the staged record buffer).
#include "engine.hpp"
#include "engine_launch.hpp"
#include "stream_io.hpp"
#include "tiles.hpp"

namespace mezo {

// The 16-byte groups a lane owns in one tile, as loaded from memory. A group
// that runs past the end of its tensor is not loaded here (it stays zero) and
// is read element by element when the tile is processed.
template <int kGroups>
struct TileRaw {
    uint4 g[kGroups];
};

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

template <int kGroups>
__device__ __forceinline__ void store_group_full(uint64_t dst, uint64_t tile, int g, uint4 v)
{
    // a buffer store over the tile's 4 KiB with the cache policy "sc1 nt"
    // (paired against "nt" alone: the 125M fp32 sweep 1.9% faster, the bf16
    // sweeps and the record loops unchanged)
    const __amdgpu_buffer_rsrc_t r = tile_rsrc(dst + tile * (kThreads * kGroups * 16), kThreads * kGroups * 16);
    store_tile_b128(r, (uint32_t(g * kThreads) + threadIdx.x) * 16u, v);
}

// Whether every step of the call is one record (a perturbation, or a restore
// and the next perturbation in one pass) and the Gaussian is the fast one:
// each record's noise then assigns the accumulators (assign4_fast) instead of
// being added to cleared ones.
template <bool kInline, bool kPortable>
__device__ __forceinline__ bool single_record_steps(const EngineArgs& a)
{
    if constexpr (!kInline || kPortable)
        return false;
    else
        return a.n_rec == 1 || (a.n_rec == 2 && a.inl[0].last);
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
    if (single_record_steps<kInline, kPortable>(a)) {
        const auto step = [&](const SeedRec& rec) {
            const SeedUniform u = seed_uniform(rec, d.tensor_id);
#pragma unroll
            for (int g = 0; g < kGroups; ++g) {
                uint32_t w0, w1, w2, w3;
                philox_words(u, pre[g], w0, w1, w2, w3);
                assign4_fast(rec.coef, w0, w1, w2, w3, acc[g][0], acc[g][1], acc[g][2], acc[g][3]);
#pragma unroll
                for (int j = 0; j < 4; ++j) th[g][j] = th[g][j] + acc[g][j];
            }
        };
        step(a.inl[0]);
        if (a.n_rec == 2) step(a.inl[1]);
    } else {
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
    if (single_record_steps<kInline, kPortable>(a)) {
        const auto step = [&](const SeedRec& rec) {
            const SeedUniform u = seed_uniform(rec, d.tensor_id);
#pragma unroll
            for (int g = 0; g < kGroups; ++g)
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    uint32_t w0, w1, w2, w3;
                    philox_words(u, pre[g][h], w0, w1, w2, w3);
                    assign4_fast(rec.coef, w0, w1, w2, w3, acc[g][4 * h + 0], acc[g][4 * h + 1], acc[g][4 * h + 2],
                                 acc[g][4 * h + 3]);
                }
            step_end();
        };
        step(a.inl[0]);
        if (a.n_rec == 2) step(a.inl[1]);
        return;
    }
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

template <bool kInline, uint32_t kDtype, bool kPortable>
__global__ __launch_bounds__(kThreads) void engine_kernel(EngineArgs a)
{
    const uint64_t tile = blockIdx.x;  // the grid is exactly the tiles of this table
    const uint32_t ti = a.tile_tensor[tile];
    const TensorDesc d = a.tensors[ti];
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

namespace {
// Launch a one-argument kernel and return the status of this launch itself
// (not the thread's last HIP error, which may hold an earlier failure of
// another caller's call).
hipError_t launch1(void (*kernel)(EngineArgs), dim3 g, dim3 b, hipStream_t stream, EngineArgs arg)
{
    void* params[] = {&arg};
    return hipLaunchKernel(reinterpret_cast<const void*>(kernel), g, b, params, 0, stream);
}

template <bool kInline, bool kPortable>
hipError_t launch_dtype(const EngineArgs& args, uint32_t dtype, dim3 g, dim3 b, hipStream_t stream)
{
    if (dtype == kF32) return launch1(engine_kernel<kInline, kF32, kPortable>, g, b, stream, args);
    return launch1(engine_kernel<kInline, kBF16, kPortable>, g, b, stream, args);
}
}  // namespace

hipError_t launch_engine_dense(const EngineArgs& args, uint32_t dtype, bool portable, hipStream_t stream)
{
    if (args.total_tiles == 0) return hipSuccess;
    if (args.total_tiles > uint64_t(0x7FFFFFFF) || (dtype != kF32 && dtype != kBF16)) return hipErrorInvalidValue;
    const bool inl = args.n_rec <= kInlineRecs;
    const dim3 g{uint32_t(args.total_tiles)};
    const dim3 b{uint32_t(kThreads)};
    if (inl)
        return portable ? launch_dtype<true, true>(args, dtype, g, b, stream)
                        : launch_dtype<true, false>(args, dtype, g, b, stream);
    return portable ? launch_dtype<false, true>(args, dtype, g, b, stream)
                    : launch_dtype<false, false>(args, dtype, g, b, stream);
}

}  // namespace mezo
