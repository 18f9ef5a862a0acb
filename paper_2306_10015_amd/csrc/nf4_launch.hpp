// nf4_launch.hpp — interface between the C-ABI host code (api.cpp) and the
// standalone NF4 conversion kernels (nf4_convert.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mezo {

// Standalone NF4 conversion of n elements between a fp32/bf16 array and NF4
// codes + absmax (device addresses).
struct NF4ConvArgs {
    uint64_t values;  // fp32 or bf16 elements
    uint64_t codes;
    uint64_t absmax;
    uint64_t n;
    uint32_t dtype;   // kF32 or kBF16 (of values)
};

// values -> NF4 (quantize) or NF4 -> values.
hipError_t launch_nf4(const NF4ConvArgs& args, bool quantize, hipStream_t stream);

}  // namespace mezo
