// launch.hpp — interface between the C-ABI host code (api.cpp) and the
// kernels (kernels.hip).
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

struct ChecksumArgs {
    const TensorDesc* tensors;
    const uint32_t* tile_tensor;
    uint64_t total_tiles;
    unsigned long long* out;  // device, accumulated with atomic adds
};

struct GenArgs {
    SeedRec rec;
    uint64_t first;
    uint64_t count;
    uint32_t* words;
    float* z;
    uint32_t tensor_id;
    uint32_t portable;  // 1: the portable Gaussian
};

// Standalone NF4 conversion of n elements between a fp32/bf16 array and NF4
// codes + absmax (device addresses).
struct NF4ConvArgs {
    uint64_t values;  // fp32 or bf16 elements
    uint64_t codes;
    uint64_t absmax;
    uint64_t n;
    uint32_t dtype;   // kF32 or kBF16 (of values)
};

// Launch the engine over the tensors of one storage type (dtype): one
// workgroup per tile (at most 2^31 - 1 tiles); portable selects the Gaussian
// made of binary32 operations only.
hipError_t launch_engine(const EngineArgs& args, uint32_t dtype, bool portable, hipStream_t stream);
hipError_t launch_generate(const GenArgs& args, hipStream_t stream);

// values -> NF4 (quantize) or NF4 -> values.
hipError_t launch_nf4(const NF4ConvArgs& args, bool quantize, hipStream_t stream);

// Zero *out, then add the checksum of every table given (one launch each).
hipError_t launch_checksum(const ChecksumArgs* tables, const uint32_t* dtypes, int n_tables,
                           unsigned long long* out, int device, hipStream_t stream);

}  // namespace mezo
