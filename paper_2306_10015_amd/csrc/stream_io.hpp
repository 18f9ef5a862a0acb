// stream_io.hpp — how the kernels stream parameter memory on gfx950: global
// address space pointer types, non-temporal 16-byte loads and stores, and
// whole-tile stores through a buffer resource with the "sc1 nt" cache policy.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mezo {

// Parameter memory is global memory; saying so lets the compiler use global_*
// instead of flat_* instructions for addresses read from the tensor table.
#define MEZO_GLOBAL __attribute__((address_space(1)))
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef MEZO_GLOBAL u32x4_t gu32x4_t;
typedef MEZO_GLOBAL float gfloat_t;
typedef MEZO_GLOBAL uint16_t gu16_t;

// Every parameter is touched once per call, so its traffic should not
// displace anything in the caches: non-temporal loads and stores.
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

// Cache-policy bits of a buffer store on gfx950: sc1 (16) | nt (2).
constexpr int kStorePolicy = 16 | 2;

// A buffer resource over [base, base + bytes) of global memory (raw buffer,
// no swizzle, default data format).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(uint64_t base, int bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(base), (short)0, bytes, 0x00020000);
}

// 16 bytes at byte offset off of a tile's buffer resource, with the "sc1 nt"
// policy (a streaming probe moved 1-2% more bytes with it than with "nt"
// alone).
__device__ __forceinline__ void store_tile_b128(__amdgpu_buffer_rsrc_t r, uint32_t off, uint4 v)
{
    const u32x4_t w = {v.x, v.y, v.z, v.w};
    __builtin_amdgcn_raw_buffer_store_b128(w, r, off, 0, kStorePolicy);
}

}  // namespace mezo
