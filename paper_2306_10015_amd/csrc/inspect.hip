// inspect.hip — inspection kernels (not on the hot path): the RNG words and
// Gaussians of an element range, and the Gaussian transform applied to given
// Philox words, so that it can be checked over chosen inputs, e.g. every one
// of the 2^24 values of u1 and of u2.
#include "engine.hpp"
#include "inspect.hpp"

namespace mezo {

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
        // the status of this launch itself, not the thread's last HIP error
        void* params[] = {&a};
        const hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(generate_kernel), dim3(uint32_t(grid)),
                                             dim3(kThreads), params, 0, stream);
        if (e != hipSuccess) return e;
        left -= n;
        first += n;
        done += n;
    }
    return hipSuccess;
}

}  // namespace mezo
