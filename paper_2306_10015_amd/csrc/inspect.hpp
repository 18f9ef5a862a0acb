// inspect.hpp — host interface of the inspection kernels (inspect.hip): the
// RNG words and Gaussians of an element range, and the Gaussian transform on
// given words. Not on the hot path.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "records.hpp"

namespace mezo {

struct GenArgs {
    SeedRec rec;
    uint64_t first;
    uint64_t count;
    uint32_t* words;
    float* z;
    uint32_t tensor_id;
    uint32_t portable;  // 1: the portable Gaussian
};

// Words and/or z of elements [first, first + count) of tensor tensor_id.
hipError_t launch_generate(const GenArgs& args, hipStream_t stream);

// z of n_blocks blocks of 4 given words (device arrays, 16-byte aligned);
// portable selects the Gaussian made of binary32 operations only.
hipError_t launch_box_muller(const uint32_t* words, uint64_t n_blocks, uint32_t portable, float* z,
                             hipStream_t stream);

}  // namespace mezo
