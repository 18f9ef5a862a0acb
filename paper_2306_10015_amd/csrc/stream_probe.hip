// stream_probe.hip — what HBM delivers to an in-place sweep with no RNG work:
// the memory ceiling the perturb sweeps are measured against.
//
// Measurement infrastructure, not part of the engine (built into
// libstream_probe.so, used by the benchmark): stream_rmw_kernel reads and
// writes a buffer in place with 16-byte accesses, an xor with a key per word
// (0 keeps every bit), in the engine's tile shape by default (256 lanes, one
// 16-byte group per lane), with the fastest cache policy found for such a
// stream, the engine's own: non-temporal loads ("nt") and stores through a
// buffer resource over the tile with "sc1 nt". (A sweep of the load policy,
// sc0 / sc1 / nt in all combinations, found only "nt" to matter; "sc1 nt"
// stores moved 1.1% and 2.4% more bytes than "nt" stores on 0.99 and 26.6 GB
// buffers.) A buffer resource also bounds the last tile: its accesses past the
// end read zero and write nothing.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kNT = 2, kSC1 = 16;  // cache-policy bits of a buffer access on gfx950

template <int kGroups, int kLanes>
__global__ __launch_bounds__(kLanes) void stream_rmw_kernel(uint64_t addr, uint64_t n_groups, uint32_t key)
{
    constexpr uint64_t kTileGroups = uint64_t(kLanes) * kGroups;
    const uint64_t first = uint64_t(blockIdx.x) * kTileGroups;  // < n_groups: the grid covers the buffer
    const uint64_t left = n_groups - first;
    const int bytes = int(16 * (left < kTileGroups ? left : kTileGroups));
    const __amdgpu_buffer_rsrc_t r =
        __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(addr + 16 * first), (short)0, bytes, 0x00020000);
    u32x4_t v[kGroups];
#pragma unroll
    for (int g = 0; g < kGroups; ++g)
        v[g] = __builtin_amdgcn_raw_buffer_load_b128(r, 16u * (uint32_t(g) * kLanes + threadIdx.x), 0, kNT);
#pragma unroll
    for (int g = 0; g < kGroups; ++g) {
        v[g] ^= key;
        __builtin_amdgcn_raw_buffer_store_b128(v[g], r, 16u * (uint32_t(g) * kLanes + threadIdx.x), 0, kSC1 | kNT);
    }
}

}  // namespace

// Enqueue one pass of stream_rmw_kernel<groups_per_lane (1 or 2), lanes (128,
// 256 or 512 per workgroup)> over the first nbytes (a multiple of 16) of data
// (16-byte aligned device memory) on stream. The last tile's buffer resource
// ends at the buffer's end. Returns 0, -1 for bad arguments, or a negative
// HIP error code.
extern "C" __attribute__((visibility("default"))) int stream_rmw(void* data, uint64_t nbytes, uint32_t key,
                                                                 int groups_per_lane, int lanes, void* stream)
{
    if (!data || (nbytes & 15u) || (reinterpret_cast<uintptr_t>(data) & 15u)) return -1;
    if (groups_per_lane != 1 && groups_per_lane != 2) return -1;
    if (lanes != 128 && lanes != 256 && lanes != 512) return -1;
    const uint64_t groups = nbytes / 16;
    const uint64_t per_tile = uint64_t(lanes) * uint64_t(groups_per_lane);
    const uint64_t tiles = (groups + per_tile - 1) / per_tile;
    if (tiles == 0 || tiles > 0x7FFFFFFFull) return -1;
    uint64_t addr = reinterpret_cast<uint64_t>(data);
    uint64_t n = groups;
    void* params[] = {&addr, &n, &key};
    const void* fn = nullptr;
    if (groups_per_lane == 1)
        fn = lanes == 128 ? reinterpret_cast<const void*>(stream_rmw_kernel<1, 128>)
           : lanes == 256 ? reinterpret_cast<const void*>(stream_rmw_kernel<1, 256>)
                          : reinterpret_cast<const void*>(stream_rmw_kernel<1, 512>);
    else
        fn = lanes == 128 ? reinterpret_cast<const void*>(stream_rmw_kernel<2, 128>)
           : lanes == 256 ? reinterpret_cast<const void*>(stream_rmw_kernel<2, 256>)
                          : reinterpret_cast<const void*>(stream_rmw_kernel<2, 512>);
    const hipError_t e = hipLaunchKernel(fn, dim3(uint32_t(tiles)), dim3(uint32_t(lanes)), params, 0,
                                         static_cast<hipStream_t>(stream));
    return e == hipSuccess ? 0 : -int(e);
}
