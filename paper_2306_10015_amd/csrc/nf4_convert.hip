// nf4_convert.hip — standalone conversions between fp32/bf16 arrays and 4-bit
// NF4 storage (codes + per-block absmax), four 2048-element tiles per
// workgroup: the forward pass of the 4-bit variant (Section 3) reads
// dequantized weights.
#include "nf4_launch.hpp"
#include "nf4_ops.hpp"

namespace mezo {

// Tiles per workgroup: a workgroup issues the loads of all its tiles before
// converting any, so that one memory latency covers several tiles (with one
// tile per workgroup the conversions waited on it: bf16 both ways about 20%
// slower).
constexpr uint32_t kQuantTiles = 4;
constexpr uint32_t kDequantTiles = 4;

// A lane's 8 input values of a quantization tile (kFull: all exist).
template <bool kFull>
__device__ __forceinline__ void nf4_quantize_load(const NF4ConvArgs& a, uint64_t e0, uint32_t valid, float (&w)[8])
{
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
}

// Whole fp32 tiles: a lane's 8 consecutive values are 32 bytes, and loading
// them as two 16-byte loads 16 bytes apart leaves every load instruction
// touching each cache line it reaches only half. So wave v loads its 512
// values of a tile (bytes [2048 v, 2048 v + 2048)) as two fully coalesced
// 16-byte loads per lane (bytes 16 l and 1024 + 16 l of that range) and hands
// them to their lanes through 2 KB of LDS of its own: every lane writes its
// two chunks and reads back the two at 32 l and 32 l + 16. A wave's LDS
// accesses complete in the order issued, so the wave needs no barrier with
// the others; the wavefront-scope fences keep the compiler from moving the
// accesses across each other. 0.169 -> 0.155 ms for the loads alone on the
// 206M-element embedding (paired).
struct QuantStage {
    u32x4_t chunk[128];  // one wave's 512 fp32 values of a tile
};

__device__ __forceinline__ void wave_lds_order()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// The two coalesced chunks of lane l of wave v of tile `tile` (whole tiles).
__device__ __forceinline__ void quantize_load_f32_coalesced(const NF4ConvArgs& a, uint64_t tile, u32x4_t& c0,
                                                            u32x4_t& c1)
{
    const uint32_t lane = threadIdx.x & 63u, wave = threadIdx.x >> 6;
    const gu32x4_t* base = reinterpret_cast<const gu32x4_t*>(a.values + (tile * kTileNF4 + wave * 512u) * 4u);
    c0 = __builtin_nontemporal_load(base + lane);
    c1 = __builtin_nontemporal_load(base + 64u + lane);
}

// Chunks -> the lane's 8 consecutive values, through the wave's stage.
__device__ __forceinline__ void quantize_exchange_f32(QuantStage& st, u32x4_t c0, u32x4_t c1, float (&w)[8])
{
    const uint32_t lane = threadIdx.x & 63u;
    wave_lds_order();  // the previous tile's reads of the stage come first
    st.chunk[lane] = c0;
    st.chunk[64u + lane] = c1;
    wave_lds_order();
    const u32x4_t r0 = st.chunk[2u * lane];
    const u32x4_t r1 = st.chunk[2u * lane + 1u];
    const uint32_t u[8] = {r0.x, r0.y, r0.z, r0.w, r1.x, r1.y, r1.z, r1.w};
#pragma unroll
    for (int j = 0; j < 8; ++j) w[j] = __uint_as_float(u[j]);
}

// Standalone quantization: kQuantTiles tiles of 2048 elements per workgroup.
__global__ __launch_bounds__(kThreads) void nf4_quantize_kernel(NF4ConvArgs a)
{
    // one copy of the round-to-nearest bin table per wave (the bin from one
    // fma, as in the engine's short calls): a wave fills its own and reads it
    // after its writes (one wave's LDS accesses complete in order), so the
    // waves of a workgroup never wait for each other
    __shared__ NF4Bin wave_bins[kThreads / 64][kNF4RoundBins];
    NF4Bin* bins = wave_bins[threadIdx.x >> 6];
    const uint32_t lane = threadIdx.x & 63u;
    bins[lane] = kNF4RoundTable.bin[lane];
    bins[lane + 64] = kNF4RoundTable.bin[lane + 64];
    if (lane == 0) bins[128] = kNF4RoundTable.bin[128];
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const uint64_t t0 = uint64_t(blockIdx.x) * kQuantTiles;
    const uint64_t lane_e = threadIdx.x * 8u;
    if ((t0 + kQuantTiles) * kTileNF4 <= a.n && a.dtype == kF32) {  // uniform: whole fp32 tiles
        __shared__ QuantStage stage[kThreads / 64];
        u32x4_t c0[kQuantTiles], c1[kQuantTiles];
#pragma unroll
        for (uint32_t t = 0; t < kQuantTiles; ++t) quantize_load_f32_coalesced(a, t0 + t, c0[t], c1[t]);
#pragma unroll
        for (uint32_t t = 0; t < kQuantTiles; ++t) {
            float w[8];
            quantize_exchange_f32(stage[threadIdx.x >> 6], c0[t], c1[t], w);
            uint32_t packed;
            float am;
            nf4_requant_round<false>(bins, 0xFFu, w, packed, am);
            nf4_store<true>(a.codes, a.absmax, (t0 + t) * kTileNF4 + lane_e, a.n, packed, am);
        }
    } else if ((t0 + kQuantTiles) * kTileNF4 <= a.n) {  // uniform: whole bf16 tiles
        float w[kQuantTiles][8];
#pragma unroll
        for (uint32_t t = 0; t < kQuantTiles; ++t) nf4_quantize_load<true>(a, (t0 + t) * kTileNF4 + lane_e, 0xFFu, w[t]);
#pragma unroll
        for (uint32_t t = 0; t < kQuantTiles; ++t) {
            uint32_t packed;
            float am;
            nf4_requant_round<false>(bins, 0xFFu, w[t], packed, am);
            nf4_store<true>(a.codes, a.absmax, (t0 + t) * kTileNF4 + lane_e, a.n, packed, am);
        }
    } else {
        for (uint32_t t = 0; t < kQuantTiles && (t0 + t) * kTileNF4 < a.n; ++t) {
            const uint64_t e0 = (t0 + t) * kTileNF4 + lane_e;
            const uint32_t valid = nf4_valid(e0, a.n);
            float w[8];
            nf4_quantize_load<false>(a, e0, valid, w);
            uint32_t packed;
            float am;
            nf4_requant_round<false>(bins, valid, w, packed, am);
            nf4_store(a.codes, a.absmax, e0, a.n, packed, am);
        }
    }
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

// A lane's 8 dequantized values of tile `tile` to the output (kFull: the
// tile is whole).
template <bool kFull>
__device__ __forceinline__ void nf4_dequantize_store(const NF4ConvArgs& a, uint64_t tile, uint64_t e0, uint32_t valid,
                                                     const float (&w)[8])
{
    if (a.dtype == kF32) {
        gfloat_t* out = reinterpret_cast<gfloat_t*>(a.values);
        if constexpr (kFull) {
            // the tile's 8 KiB of output through a buffer resource, with the
            // engine's store policy
            const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
                reinterpret_cast<void*>(a.values + tile * kTileNF4 * 4), (short)0, int(kTileNF4 * 4), 0x00020000);
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
                reinterpret_cast<void*>(a.values + tile * kTileNF4 * 2), (short)0, int(kTileNF4 * 2), 0x00020000);
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

// Standalone dequantization: kDequantTiles tiles of 2048 elements per workgroup.
__global__ __launch_bounds__(kThreads) void nf4_dequantize_kernel(NF4ConvArgs a)
{
    const uint32_t table = nf4_value_lanes();
    const uint64_t t0 = uint64_t(blockIdx.x) * kDequantTiles;
    const uint64_t lane_e = threadIdx.x * 8u;
    if (a.dtype == kF32 && (t0 + kDequantTiles) * kTileNF4 <= a.n) {
        // fp32 output: each tile as two halves of 1024 elements, lane l taking
        // elements 4l .. 4l + 3 of each, so that every 16-byte store is
        // contiguous across the lanes and writes whole cache lines (a lane's 8
        // consecutive elements as two 16-byte stores leave every line half
        // written by each store, which ran 4.5x slower with streaming stores)
        uint32_t code16[kDequantTiles][2];
        float am[kDequantTiles][2];
        const uint64_t lane4 = threadIdx.x * 4u;
#pragma unroll
        for (uint32_t t = 0; t < kDequantTiles; ++t)
#pragma unroll
            for (uint32_t h = 0; h < 2; ++h) {
                const uint64_t e = (t0 + t) * kTileNF4 + h * (kTileNF4 / 2) + lane4;
                code16[t][h] = __builtin_nontemporal_load(reinterpret_cast<const gu16_t*>(a.codes + e / 2));
                am[t][h] = reinterpret_cast<const gfloat_t*>(a.absmax)[e / kNF4Block];
            }
#pragma unroll
        for (uint32_t t = 0; t < kDequantTiles; ++t) {
            const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
                reinterpret_cast<void*>(a.values + (t0 + t) * kTileNF4 * 4), (short)0, int(kTileNF4 * 4), 0x00020000);
#pragma unroll
            for (uint32_t h = 0; h < 2; ++h) {
                uint32_t v[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int addr = int(((code16[t][h] >> (4 * j)) & 15u) << 2);
                    v[j] = __float_as_uint(__uint_as_float(uint32_t(__builtin_amdgcn_ds_bpermute(addr, int(table))))
                                           * am[t][h]);
                }
                const u32x4_t q = {v[0], v[1], v[2], v[3]};
                __builtin_amdgcn_raw_buffer_store_b128(q, r, h * (kTileNF4 / 2) * 4 + threadIdx.x * 16u, 0,
                                                       kStorePolicy);
            }
        }
    } else if ((t0 + kDequantTiles) * kTileNF4 <= a.n) {  // uniform: all the workgroup's tiles are whole
        uint32_t packed[kDequantTiles];
        float am[kDequantTiles];
#pragma unroll
        for (uint32_t t = 0; t < kDequantTiles; ++t)
            nf4_load<true>(a.codes, a.absmax, (t0 + t) * kTileNF4 + lane_e, a.n, packed[t], am[t]);
#pragma unroll
        for (uint32_t t = 0; t < kDequantTiles; ++t) {
            float w[8];
            nf4_dequant_lanes(table, packed[t], am[t], 0xFFu, w);
            nf4_dequantize_store<true>(a, t0 + t, (t0 + t) * kTileNF4 + lane_e, 0xFFu, w);
        }
    } else {
        for (uint32_t t = 0; t < kDequantTiles && (t0 + t) * kTileNF4 < a.n; ++t) {
            const uint64_t e0 = (t0 + t) * kTileNF4 + lane_e;
            const uint32_t valid = nf4_valid(e0, a.n);
            uint32_t packed;
            float am;
            nf4_load(a.codes, a.absmax, e0, a.n, packed, am);
            float w[8];
            nf4_dequant_lanes(table, packed, am, valid, w);
            nf4_dequantize_store<false>(a, t0 + t, e0, valid, w);
        }
    }
}

hipError_t launch_nf4(const NF4ConvArgs& args, bool quantize, hipStream_t stream)
{
    const uint64_t tiles = (args.n + kTileNF4 - 1) / kTileNF4;
    if (tiles == 0) return hipSuccess;
    const uint64_t per = quantize ? kQuantTiles : kDequantTiles;
    const uint64_t groups = (tiles + per - 1) / per;
    if (groups > uint64_t(0x7FFFFFFF)) return hipErrorInvalidValue;
    const dim3 g{uint32_t(groups)};
    const dim3 b{uint32_t(kThreads)};
    NF4ConvArgs arg = args;
    void* params[] = {&arg};
    return hipLaunchKernel(reinterpret_cast<const void*>(quantize ? nf4_quantize_kernel : nf4_dequantize_kernel), g,
                           b, params, 0, stream);
}

}  // namespace mezo
