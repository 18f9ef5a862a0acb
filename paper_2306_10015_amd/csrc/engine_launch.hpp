// engine_launch.hpp — interface between the C-ABI host code (api.cpp) and the
// engine kernels (engine_dense.hip: fp32 and bf16 storage; engine_nf4.hip:
// 4-bit storage).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "records.hpp"

namespace mezo {

// Kernel arguments of the engine kernel, one launch per storage type. Up to
// kInlineRecs records travel in the arguments themselves; longer lists are
// staged in device memory (ext).
struct EngineArgs {
    const TensorDesc* tensors;     // device table of one storage type, tile_begin ascending
    const uint32_t* tile_tensor;   // device: index into tensors of every tile
    const TensorDesc* src_tensors; // device table to read from (same layout), or null: in place
    uint64_t total_tiles;
    const SeedRec* ext;         // device records when n_rec > kInlineRecs
    uint32_t n_tensors;
    uint32_t n_rec;
    SeedRec inl[kInlineRecs];
};

// Launch the engine over the tensors of one storage type: one workgroup per
// tile (at most 2^31 - 1 tiles); portable selects the Gaussian made of
// binary32 operations only. dtype is kF32 or kBF16 for launch_engine_dense.
hipError_t launch_engine_dense(const EngineArgs& args, uint32_t dtype, bool portable, hipStream_t stream);
hipError_t launch_engine_nf4(const EngineArgs& args, bool portable, hipStream_t stream);

}  // namespace mezo
