// noalloc_launch.hpp — interface between the C-ABI host code (api.cpp) and the
// record staging of the entry point that allocates nothing (noalloc.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "records.hpp"

namespace mezo {

// Records the file-scope staging array holds: 65536 x 32 B = 2 MiB per GPU.
constexpr uint32_t kNoAllocRecords = 65536;
// Records one staging launch carries in its arguments.
constexpr uint32_t kStageRecs = 32;

struct StageArgs {
    SeedRec* dst;      // the staging array's device address on the current device
    uint32_t offset;   // index of recs[0] in it
    uint32_t n;        // records in recs, 1 .. kStageRecs
    SeedRec recs[kStageRecs];
};

// The device address of the staging array on the current device (found once
// per device with hipGetSymbolAddress; no allocation).
hipError_t noalloc_scratch(SeedRec** out);

// Enqueue a copy of n records (1 .. kStageRecs, taken into the kernel
// arguments before this returns) to dst[offset ..] on stream.
hipError_t launch_stage(SeedRec* dst, uint32_t offset, const SeedRec* recs, uint32_t n, hipStream_t stream);

}  // namespace mezo
