// checksum_launch.hpp — interface between the C-ABI host code (api.cpp) and
// the checksum kernels (checksum.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "records.hpp"

namespace mezo {

struct ChecksumArgs {
    const TensorDesc* tensors;
    const uint32_t* tile_tensor;
    uint64_t total_tiles;
    unsigned long long* out;  // device, accumulated with atomic adds
};

// Zero *out, then add the checksum of every table given (one launch each).
hipError_t launch_checksum(const ChecksumArgs* tables, const uint32_t* dtypes, int n_tables,
                           unsigned long long* out, int device, hipStream_t stream);

}  // namespace mezo
