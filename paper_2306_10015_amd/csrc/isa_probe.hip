// isa_probe.hip — issue cost of the VALU instructions the engine's inner loop
// is made of, measured on the device the benchmark runs on (gfx950).
//
// Measurement infrastructure for the benchmark's ALU roofline, not part of
// the engine: libisa_probe.so exports one C function. Each probe kernel runs,
// per lane, kChains independent dependency chains of one instruction for
// kIter iterations at full occupancy (8 waves per SIMD); the cost reported is
// SIMD cycles per wave instruction at 2.4 GHz (a full-rate instruction on a
// 16-lane SIMD takes 4). Every lane writes one word into a buffer sized for the
// whole grid, so every access is in bounds.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int kIter = 2048;
constexpr int kChains = 8;

#define PROBE_U32(name, body)                                                     \
    __global__ __launch_bounds__(256) void name(uint32_t* out, uint32_t s)        \
    {                                                                             \
        uint32_t x[kChains];                                                      \
        for (int i = 0; i < kChains; ++i) x[i] = threadIdx.x * (i + 1) + s;       \
        for (int it = 0; it < kIter; ++it)                                        \
            for (int i = 0; i < kChains; ++i) { body; }                           \
        uint32_t r = 0;                                                           \
        for (int i = 0; i < kChains; ++i) r ^= x[i];                              \
        out[blockIdx.x * blockDim.x + threadIdx.x] = r;                           \
    }

#define PROBE_F32(name, body)                                                     \
    __global__ __launch_bounds__(256) void name(uint32_t* out, uint32_t s)        \
    {                                                                             \
        float x[kChains];                                                         \
        for (int i = 0; i < kChains; ++i) x[i] = 0.1f + 1e-6f * (threadIdx.x * (i + 1) + s); \
        for (int it = 0; it < kIter; ++it)                                        \
            for (int i = 0; i < kChains; ++i) { body; }                           \
        float r = 0.0f;                                                           \
        for (int i = 0; i < kChains; ++i) r += x[i];                              \
        out[blockIdx.x * blockDim.x + threadIdx.x] = __float_as_uint(r);          \
    }

__global__ __launch_bounds__(256) void p_mad_u64(uint32_t* out, uint32_t s)
{
    uint64_t x[kChains];
    for (int i = 0; i < kChains; ++i) x[i] = threadIdx.x * (i + 1) + s;
    for (int it = 0; it < kIter; ++it)
        for (int i = 0; i < kChains; ++i)
            asm volatile("v_mad_u64_u32 %0, vcc, %1, %2, %0"
                         : "+v"(x[i]) : "v"(uint32_t(x[i])), "s"(0xD2511F53u) : "vcc");
    uint32_t r = 0;
    for (int i = 0; i < kChains; ++i) r ^= uint32_t(x[i]) ^ uint32_t(x[i] >> 32);
    out[blockIdx.x * blockDim.x + threadIdx.x] = r;
}
PROBE_U32(p_bitop3, asm volatile("v_bitop3_b32 %0, %0, %1, %2 bitop3:0x96" : "+v"(x[i]) : "v"(s + i), "s"(s));)
PROBE_U32(p_xor, asm volatile("v_xor_b32 %0, %1, %0" : "+v"(x[i]) : "v"(s + i));)
PROBE_U32(p_lshr, asm volatile("v_lshrrev_b32 %0, 1, %0" : "+v"(x[i]));)
PROBE_U32(p_cvt, asm volatile("v_cvt_f32_u32 %0, %0" : "+v"(x[i]));)
PROBE_F32(p_fma, asm volatile("v_fma_f32 %0, %0, %1, %1" : "+v"(x[i]) : "v"(0.5f));)
PROBE_F32(p_fmac, asm volatile("v_fmac_f32 %0, %1, %2" : "+v"(x[i]) : "v"(0.5f), "v"(0.25f));)
PROBE_F32(p_fmamk, asm volatile("v_fmamk_f32 %0, %0, 0x33800000, %1" : "+v"(x[i]) : "v"(0.5f));)
PROBE_F32(p_mul, asm volatile("v_mul_f32 %0, %0, %1" : "+v"(x[i]) : "v"(0.999f));)
PROBE_F32(p_add, asm volatile("v_add_f32 %0, %0, %1" : "+v"(x[i]) : "v"(0.5f));)
PROBE_F32(p_log, asm volatile("v_log_f32 %0, %0" : "+v"(x[i]));)
PROBE_F32(p_sqrt, asm volatile("v_sqrt_f32 %0, %0" : "+v"(x[i]));)
PROBE_F32(p_sin, asm volatile("v_sin_f32 %0, %0" : "+v"(x[i]));)
PROBE_F32(p_cos, asm volatile("v_cos_f32 %0, %0" : "+v"(x[i]));)
PROBE_U32(p_mov, asm volatile("v_mov_b32 %0, %1" : "=v"(x[i]) : "v"(x[(i + 1) % kChains]));)

// In-place streaming read-modify-write with the engine's access pattern: one
// kLanes-lane workgroup per tile of kGroups 16-byte groups per lane, the
// groups strided by kLanes, non-temporal loads and stores, and one xor per
// 32-bit word with a runtime key as the only arithmetic (key 0 leaves every
// bit as it was): the memory ceiling of a sweep.
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

typedef void (*probe_fn)(uint32_t*, uint32_t);

struct Probe {
    const char* name;
    probe_fn fn;
};

const Probe kProbes[] = {
    {"v_mad_u64_u32", p_mad_u64}, {"v_bitop3_b32", p_bitop3}, {"v_xor_b32", p_xor},
    {"v_lshrrev_b32", p_lshr},    {"v_cvt_f32_u32", p_cvt},   {"v_fma_f32", p_fma},
    {"v_fmac_f32", p_fmac},       {"v_fmamk_f32", p_fmamk},     {"v_mul_f32", p_mul},       {"v_add_f32", p_add},
    {"v_log_f32", p_log},         {"v_sqrt_f32", p_sqrt},     {"v_sin_f32", p_sin},
    {"v_cos_f32", p_cos},         {"v_mov_b32", p_mov},
};

}  // namespace

extern "C" __attribute__((visibility("default"))) int isa_probe_count(void)
{
    return int(sizeof(kProbes) / sizeof(kProbes[0]));
}

extern "C" __attribute__((visibility("default"))) const char* isa_probe_name(int i)
{
    return (i >= 0 && i < isa_probe_count()) ? kProbes[i].name : "";
}

// cycles[i] = SIMD cycles per wave instruction of probe i at clock_ghz.
// Returns 0, or a negative HIP error code.
extern "C" __attribute__((visibility("default"))) int isa_probe_run(double* cycles, double clock_ghz)
{
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess) return -1;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return -1;
    const int block = 256, grid = cus * 8;  // 8 workgroups of 4 waves per CU: 8 waves per SIMD
    uint32_t* out = nullptr;
    if (hipMalloc(&out, sizeof(uint32_t) * size_t(grid) * block) != hipSuccess) return -2;
    hipEvent_t a = nullptr, b = nullptr;
    int rc = 0;
    if (hipEventCreate(&a) != hipSuccess || hipEventCreate(&b) != hipSuccess) rc = -3;
    for (int i = 0; rc == 0 && i < isa_probe_count(); ++i) {
        hipLaunchKernelGGL(kProbes[i].fn, dim3(grid), dim3(block), 0, 0, out, 1u);  // warm
        (void)hipEventRecord(a, 0);
        hipLaunchKernelGGL(kProbes[i].fn, dim3(grid), dim3(block), 0, 0, out, 1u);
        (void)hipEventRecord(b, 0);
        if (hipEventSynchronize(b) != hipSuccess) { rc = -4; break; }
        float ms = 0.0f;
        (void)hipEventElapsedTime(&ms, a, b);
        const double wave_instr = double(grid) * (block / 64) * kIter * kChains;
        const double simd_cycles = double(ms) * 1e-3 * clock_ghz * 1e9 * cus * 4;
        cycles[i] = simd_cycles / wave_instr;
    }
    if (a) (void)hipEventDestroy(a);
    if (b) (void)hipEventDestroy(b);
    (void)hipFree(out);
    return rc;
}

// Enqueue one pass of stream_rmw_kernel<groups_per_lane (1 or 2), lanes (128,
// 256 or 512 per workgroup)> over the first nbytes (a multiple of 16) of data
// (16-byte aligned device memory) on stream. Returns 0, -1 for bad arguments,
// or a negative HIP error code.
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
