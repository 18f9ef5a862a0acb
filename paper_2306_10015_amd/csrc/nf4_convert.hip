// nf4_convert.hip — standalone conversions between fp32/bf16 arrays and 4-bit
// NF4 storage (codes + per-block absmax), one 2048-element tile per
// workgroup: the forward pass of the 4-bit variant (Section 3) reads
// dequantized weights.
#include "nf4_launch.hpp"
#include "nf4_ops.hpp"

namespace mezo {

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

hipError_t launch_nf4(const NF4ConvArgs& args, bool quantize, hipStream_t stream)
{
    const uint64_t tiles = (args.n + kTileNF4 - 1) / kTileNF4;
    if (tiles == 0) return hipSuccess;
    if (tiles > uint64_t(0x7FFFFFFF)) return hipErrorInvalidValue;
    const dim3 g{uint32_t(tiles)};
    const dim3 b{uint32_t(kThreads)};
    NF4ConvArgs arg = args;
    void* params[] = {&arg};
    return hipLaunchKernel(reinterpret_cast<const void*>(quantize ? nf4_quantize_kernel : nf4_dequantize_kernel), g,
                           b, params, 0, stream);
}

}  // namespace mezo
