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
    unsigned long long* out;  // device: the checksum, written by the call's last launch
    // device, two words that are zero between calls: [0] the running sum
    // (64-bit atomic adds), [1] the workgroups of this launch done so far
    unsigned long long* acc;
    uint32_t last;  // 1: this launch ends the call (writes *out, clears acc[0])
};

// The checksum of every table given (one launch each) into *out, summed in
// acc (two zero words, left zero again; calls that share acc must not
// overlap in time).
hipError_t launch_checksum(const ChecksumArgs* tables, const uint32_t* dtypes, int n_tables,
                           unsigned long long* out, unsigned long long* acc, int device, hipStream_t stream);

}  // namespace mezo
