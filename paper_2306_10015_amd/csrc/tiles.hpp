// tiles.hpp — the tile decomposition of fp32 and bf16 tensors shared by the
// engine and the checksum: a workgroup of kThreads lanes takes one tile; each
// lane owns kGroups 16-byte groups of it, strided by kThreads groups so that
// every wave touches one contiguous 1 KiB run per group.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "records.hpp"

namespace mezo {

template <uint32_t kDtype>
struct Layout;
template <>
struct Layout<kF32> {
    static constexpr int kGroups = kGroupsF32;
    static constexpr uint64_t kPerGroup = 4;  // elements per 16-byte group
};
template <>
struct Layout<kBF16> {
    static constexpr int kGroups = kGroupsBF16;
    static constexpr uint64_t kPerGroup = 8;
};

// Index (within its tensor) of the g-th 16-byte group this lane owns in tile.
template <int kGroups>
__device__ __forceinline__ uint64_t group_index(uint64_t tile, int g)
{
    return tile * (kThreads * kGroups) + uint64_t(g) * kThreads + threadIdx.x;
}

}  // namespace mezo
