// noalloc.hip — the record staging of the entry point that allocates nothing
// (mezo_replay_noalloc): a file-scope device array holds a call's records,
// written by small kernels that carry up to kStageRecs records each in their
// arguments (so no host buffer has to outlive the call and nothing is copied
// from host memory), and read by the engine kernel like any staged list.
//
// Every GPU the library runs on holds its own copy of the array until the
// process ends; host code reaches it only through the address
// hipGetSymbolAddress returns for the device that is current (the array's
// name in host code is a host-side stand-in, not a device address).
#include <atomic>
#include <mutex>

#include "noalloc_launch.hpp"

namespace mezo {

static __device__ __align__(256) SeedRec scratch[kNoAllocRecords];

__global__ __launch_bounds__(64) void stage_records_kernel(StageArgs a)
{
    // one record per lane; a.n <= kStageRecs <= 64 (checked on the host)
    if (threadIdx.x < a.n) a.dst[a.offset + threadIdx.x] = a.recs[threadIdx.x];
}

namespace {
constexpr int kMaxDevices = 64;
std::atomic<SeedRec*> g_scratch[kMaxDevices];
std::mutex g_scratch_mu;
}  // namespace

hipError_t noalloc_scratch(SeedRec** out)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    SeedRec* p = g_scratch[dev].load(std::memory_order_acquire);
    if (!p) {
        // once per device, with that device current
        std::lock_guard<std::mutex> lock(g_scratch_mu);
        p = g_scratch[dev].load(std::memory_order_acquire);
        if (!p) {
            void* addr = nullptr;
            e = hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch));
            if (e != hipSuccess) return e;
            if (!addr) return hipErrorInvalidSymbol;
            p = static_cast<SeedRec*>(addr);
            g_scratch[dev].store(p, std::memory_order_release);
        }
    }
    *out = p;
    return hipSuccess;
}

hipError_t launch_stage(SeedRec* dst, uint32_t offset, const SeedRec* recs, uint32_t n, hipStream_t stream)
{
    if (!dst || n == 0 || n > kStageRecs || offset > kNoAllocRecords - n) return hipErrorInvalidValue;
    StageArgs a;
    a.dst = dst;
    a.offset = offset;
    a.n = n;
    for (uint32_t i = 0; i < n; ++i) a.recs[i] = recs[i];
    void* params[] = {&a};
    // the status of this launch itself, not the thread's last HIP error
    return hipLaunchKernel(reinterpret_cast<const void*>(stage_records_kernel), dim3(1), dim3(64), params, 0,
                           stream);
}

}  // namespace mezo
