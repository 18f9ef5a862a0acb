// inspect.hpp — host interface of the inspection kernels (inspect.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mezo {

// z of n_blocks blocks of 4 given words (device arrays, 16-byte aligned);
// portable selects the Gaussian made of binary32 operations only.
hipError_t launch_box_muller(const uint32_t* words, uint64_t n_blocks, uint32_t portable, float* z,
                             hipStream_t stream);

}  // namespace mezo
