// inspect.hip — inspection kernels (not on the hot path): the Gaussian
// transform applied to given Philox words, so that it can be checked over
// chosen inputs, e.g. every one of the 2^24 values of u1 and of u2.
#include "engine.hpp"
#include "inspect.hpp"

namespace mezo {

// z of every block of 4 words: the same gauss4 / gauss4_portable the engine's
// inspection path uses (the update path applies the same pair transform with
// the coefficient folded into the radius).
__global__ __launch_bounds__(kThreads) void box_muller_kernel(const uint32_t* words, uint64_t n_blocks,
                                                              uint32_t portable, float* z)
{
    const uint64_t b = uint64_t(blockIdx.x) * kThreads + threadIdx.x;
    if (b >= n_blocks) return;
    const uint4 w = reinterpret_cast<const uint4*>(words)[b];
    const Z4 r = portable ? gauss4_portable(w.x, w.y, w.z, w.w) : gauss4(w.x, w.y, w.z, w.w);
    reinterpret_cast<float4*>(z)[b] = make_float4(r.z0, r.z1, r.z2, r.z3);
}

hipError_t launch_box_muller(const uint32_t* words, uint64_t n_blocks, uint32_t portable, float* z,
                             hipStream_t stream)
{
    // at most 2^26 blocks per launch
    const uint64_t kChunk = uint64_t(1) << 26;
    for (uint64_t done = 0; done < n_blocks; done += kChunk) {
        const uint64_t n = n_blocks - done < kChunk ? n_blocks - done : kChunk;
        const uint64_t grid = (n + kThreads - 1) / kThreads;
        const uint32_t* w = words + 4 * done;
        float* zo = z + 4 * done;
        uint64_t cnt = n;
        uint32_t pt = portable;
        // the status of this launch itself, not the thread's last HIP error
        void* params[] = {&w, &cnt, &pt, &zo};
        const hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(box_muller_kernel), dim3(uint32_t(grid)),
                                             dim3(kThreads), params, 0, stream);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace mezo
