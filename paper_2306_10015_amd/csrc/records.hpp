// records.hpp — structures and constants shared by the host code (api.cpp)
// and the kernels (*.hip): the seed record, the tensor table entry, the
// work decomposition and the Philox4x32-10 constants.
#pragma once

#include <stdint.h>

namespace mezo {

// One perturbation to apply: seed-derived Philox inputs and its weight.
// 32 bytes, read by every wave with one scalar load.
struct alignas(16) SeedRec {
    uint32_t key0;    // Philox key, low word  = low 32 bits of the machine id
    uint32_t key1;    // Philox key, high word = high 32 bits of the machine id
    uint32_t step;    // counter word 3
    uint32_t mb_hi;   // high word of kMulB * sample (round 1, counter word 2)
    uint32_t mb_lo;   // low word  of kMulB * sample
    float    coef;    // fl32(c * sqrt(2 ln 2)): the weight c of z in theta += c * z,
                      // pre-multiplied by the constant the kernel leaves out of z
    uint32_t last;    // 1: round to storage after this record (end of a step)
    uint32_t sample;  // counter word 2 (inspection only)
};

// One registered tensor as the kernels see it.
struct alignas(16) TensorDesc {
    uint64_t data;        // device address, 16-byte aligned (NF4: the codes)
    uint64_t numel;
    uint64_t tile_begin;  // first global tile of this tensor
    uint32_t tensor_id;
    uint32_t dtype;       // 0 = fp32, 1 = bf16, 2 = NF4
    uint64_t aux;         // NF4: device address of the per-block absmax values
    uint64_t first;       // index of element 0 within the logical tensor (a shard's offset)
};

constexpr uint32_t kF32 = 0u;
constexpr uint32_t kBF16 = 1u;
constexpr uint32_t kNF4 = 2u;
constexpr uint32_t kStorageTypes = 3u;

// Work decomposition: a workgroup of kThreads lanes handles one tile; each
// lane owns kGroups 16-byte groups of the tile, strided by kThreads groups so
// that every wave touches one contiguous 1 KiB run per group. A 16-byte group
// is 4 fp32 elements (one Philox block) or 8 bf16 elements (two blocks). One
// group per lane (4 KiB tiles: 1024 fp32 or 2048 bf16 elements) streams
// faster than two: more workgroups in flight per byte.
constexpr int kThreads = 256;
constexpr int kGroupsF32 = 1;
constexpr int kGroupsBF16 = 1;
constexpr uint64_t kTileF32 = uint64_t(kThreads) * kGroupsF32 * 4;
constexpr uint64_t kTileBF16 = uint64_t(kThreads) * kGroupsBF16 * 8;
// NF4: each lane owns 8 consecutive elements (4 code bytes, two Philox
// blocks); 8 lanes make one block of kNF4Block elements sharing one absmax.
constexpr uint64_t kTileNF4 = uint64_t(kThreads) * 8;
constexpr int kNF4Block = 64;

// Records that travel inside the kernel arguments (above this they are staged
// in device memory).
constexpr uint32_t kInlineRecs = 32;

// ---- Philox4x32-10 ---------------------------------------------------------
// Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as 1, 2, 3"
// (SC'11): multipliers and Weyl key increments of the 4x32 variant.
constexpr uint32_t kMulA = 0xD2511F53u;
constexpr uint32_t kMulB = 0xCD9E8D57u;
constexpr uint32_t kWeylA = 0x9E3779B9u;
constexpr uint32_t kWeylB = 0xBB67AE85u;

// ---- checksum -------------------------------------------------------------
// A tensor's bytes as little-endian 8-byte chunks c_j (the last zero-padded);
// checksum = sum over all chunks of all tensors of
// fmix64(c_j ^ j * kChunkPos ^ tensor_id * kChunkTensor) mod 2^64, fmix64 being
// MurmurHash3's 64-bit finalizer (multipliers kFmixA, kFmixB).
constexpr uint64_t kChunkPos = 0x9E3779B97F4A7C15ull;
constexpr uint64_t kChunkTensor = 0xD1B54A32D192ED03ull;
constexpr uint64_t kFmixA = 0xFF51AFD7ED558CCDull;
constexpr uint64_t kFmixB = 0xC4CEB9FE1A85EC53ull;

// sqrt(2 ln 2) in double: the engine kernels produce z / sqrt(2 ln 2) and the
// host folds the factor into every record's coefficient.
constexpr double kZScaleF64 = 1.17741002251547469101;

}  // namespace mezo
