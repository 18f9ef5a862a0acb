// stream_probe.hip — what HBM delivers to an in-place sweep with no RNG work:
// the memory ceiling the perturb sweeps are measured against.
//
// Measurement infrastructure, not part of the engine (built into
// libstream_probe.so, used by the benchmark): stream_rmw_kernel reads and
// writes a buffer in place with non-temporal 16-byte accesses, an xor with a
// key per word (0 keeps every bit), in the engine's tile shape by default (256
// lanes, one 16-byte group per lane).
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) u32x4_t gu32x4_t;

template <int kGroups, int kLanes>
__global__ __launch_bounds__(kLanes) void stream_rmw_kernel(uint64_t addr, uint64_t n_groups, uint32_t key)
{
    gu32x4_t* data = reinterpret_cast<gu32x4_t*>(addr);
    const uint64_t base = uint64_t(blockIdx.x) * (kLanes * kGroups);
#pragma unroll
    for (int g = 0; g < kGroups; ++g) {
        const uint64_t i = base + uint64_t(g) * kLanes + threadIdx.x;
        if (i < n_groups) {
            u32x4_t v = __builtin_nontemporal_load(data + i);
            v ^= key;
            __builtin_nontemporal_store(v, data + i);
        }
    }
}

}  // namespace

// Enqueue one pass of stream_rmw_kernel<groups_per_lane (1 or 2), lanes (128,
// 256 or 512 per workgroup)> over the first nbytes (a multiple of 16) of data
// (16-byte aligned device memory) on stream. Every lane checks its group
// against the buffer's end. Returns 0, -1 for bad arguments, or a negative
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
