// engine_nf4.hip — the engine kernels on 4-bit NF4 storage (gfx950): the
// same records as on fp32/bf16 storage, with the block dequantized once
// before the first record and quantized again at every step end (Section 3:
// the weights are dequantized before the noise is added and quantized again
// afterwards). Three kernels by the length of the record list: one loop over
// any number of records (engine_nf4_kernel), two records
// (engine_nf4_short_kernel) and one record, 16 elements per lane
// (engine_nf4_sweep_kernel).
#include "engine.hpp"
#include "engine_launch.hpp"
#include "nf4_ops.hpp"

namespace mezo {

// kFull: a tile wholly inside its tensor, where every lane's 8 elements exist
// (no masks, no bounds).
template <bool kInline, bool kPortable, bool kFull>
__device__ __forceinline__ void tile_nf4(const EngineArgs& a, const TensorDesc& d, uint64_t e0, uint32_t packed,
                                         float am, const NF4Lds& s)
{
    const uint32_t valid = kFull ? 0xFFu : nf4_valid(e0, d.numel);
    float w[8];
    nf4_dequant(s, packed, am, valid, w);
    float acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = 0.0f;
    const uint64_t blk = (d.first + e0) >> 2;  // block of the logical tensor
    const BlockPre pre0 = block_pre(uint32_t(blk));
    const BlockPre pre1 = block_pre(uint32_t(blk + 1));
    const auto accumulate = [&](uint32_t r) {
        const SeedRec& rec = rec_at<kInline>(a, r);
        const SeedUniform u = seed_uniform(rec, d.tensor_id);
        const float c = rec.coef;
        uint32_t w0, w1, w2, w3;
        philox_words(u, pre0, w0, w1, w2, w3);
        accumulate4<kPortable>(c, w0, w1, w2, w3, acc[0], acc[1], acc[2], acc[3]);
        philox_words(u, pre1, w0, w1, w2, w3);
        accumulate4<kPortable>(c, w0, w1, w2, w3, acc[4], acc[5], acc[6], acc[7]);
    };
    const auto step_end = [&]() {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            w[j] = w[j] + acc[j];
            acc[j] = 0.0f;
        }
        if (partial_wave(valid)) {  // only waves that reach a tensor's end
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (!((valid >> j) & 1u)) w[j] = 0.0f;
        }
    };
    if (a.n_rec == 0) {  // out of place with nothing to apply: a copy
        nf4_store<kFull>(d.data, d.aux, e0, d.numel, packed, am);
        return;
    }
    // every record list ends a step with its last record, which is peeled off
    // the loop: its quantization needs no values for a next step
    for (uint32_t r = 0; r + 1 < a.n_rec; ++r) {
        accumulate(r);
        if (rec_at<kInline>(a, r).last) {
            step_end();
            nf4_requant<true>(s.bin, valid, w, packed, am);
        }
    }
    accumulate(a.n_rec - 1);
    step_end();
    nf4_requant<false>(s.bin, valid, w, packed, am);
    nf4_store<kFull>(d.data, d.aux, e0, d.numel, packed, am);
}

// The noise of record r for a lane's 8 elements: acc = c z (kSet, a step's
// first record, which saves zeroing the accumulators; in fast mode the
// product can differ from fma(c, z, +0) only in the sign of a zero, which no
// code depends on, +0 and -0 sharing the zero code's bin) or acc += c z.
template <bool kPortable, bool kSet>
__device__ __forceinline__ void short_record(const SeedRec& rec, uint32_t tensor_id, BlockPre pre0, BlockPre pre1,
                                             float (&acc)[8])
{
    const SeedUniform u = seed_uniform(rec, tensor_id);
    const float c = rec.coef;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        uint32_t w0, w1, w2, w3;
        philox_words(u, h ? pre1 : pre0, w0, w1, w2, w3);
        float* a4 = acc + 4 * h;
        if constexpr (!kSet) {
            accumulate4<kPortable>(c, w0, w1, w2, w3, a4[0], a4[1], a4[2], a4[3]);
        } else if constexpr (kPortable) {
            const Z4 z = gauss4_portable(w0, w1, w2, w3);
            a4[0] = c * z.z0;
            a4[1] = c * z.z1;
            a4[2] = c * z.z2;
            a4[3] = c * z.z3;
        } else {
            assign4_fast(c, w0, w1, w2, w3, a4[0], a4[1], a4[2], a4[3]);
        }
    }
}

// A step of one record on a lane's 8 values: w = round(w + c z). Portable
// mode: acc = c z, then w + acc, the two roundings its definition states.
// Fast mode: w = fma(c r, cos, w) and fma(c r, sin, w), one rounding of the
// value plus the noise (as the oracle's step, a sum rounded once to binary32;
// the fast mode's z is within its tolerance either way).
template <bool kPortable>
__device__ __forceinline__ void short_step(const SeedRec& rec, uint32_t tensor_id, BlockPre pre0, BlockPre pre1,
                                           float (&w)[8])
{
    if constexpr (kPortable) {
        float acc[8];
        short_record<true, true>(rec, tensor_id, pre0, pre1, acc);
#pragma unroll
        for (int j = 0; j < 8; ++j) w[j] = w[j] + acc[j];
    } else {
        const SeedUniform u = seed_uniform(rec, tensor_id);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            uint32_t w0, w1, w2, w3;
            philox_words(u, h ? pre1 : pre0, w0, w1, w2, w3);
            box_muller_pair_acc(w0, w1, rec.coef, w[4 * h], w[4 * h + 1]);
            box_muller_pair_acc(w2, w3, rec.coef, w[4 * h + 2], w[4 * h + 3]);
        }
    }
}

// A lane's 8 elements (Philox blocks blk and blk + 1 of its tensor) through a
// call of one or two records (inline): dequantize through the pair table, the
// records, and at each step end quantize on the round-to-nearest table.
// kFull: the 8 elements all exist (no masks).
template <bool kPortable, bool kFull>
__device__ __forceinline__ void short_records(const EngineArgs& a, uint32_t tensor_id, uint32_t blk, uint32_t valid,
                                              const NF4ShortLds& s, uint32_t& packed, float& am)
{
    float w[8];
    nf4_dequant_pairs(s, packed, am, valid, w);
    const BlockPre pre0 = block_pre(blk);
    const BlockPre pre1 = block_pre(blk + 1);
    const auto mask = [&]() {
        if (!kFull && partial_wave(valid)) {  // only waves that reach a tensor's end
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (!((valid >> j) & 1u)) w[j] = 0.0f;
        }
    };
    if (a.n_rec == 2 && !a.inl[0].last) {  // two records in one step: their sum, one rounding
        float acc[8];
        short_record<kPortable, true>(a.inl[0], tensor_id, pre0, pre1, acc);
        short_record<kPortable, false>(a.inl[1], tensor_id, pre0, pre1, acc);
#pragma unroll
        for (int j = 0; j < 8; ++j) w[j] = w[j] + acc[j];
    } else {  // every step of one record
        short_step<kPortable>(a.inl[0], tensor_id, pre0, pre1, w);
        if (a.n_rec == 2) {
            mask();
            nf4_requant_round<true, kPortable>(s.bin, valid, w, packed, am);
            short_step<kPortable>(a.inl[1], tensor_id, pre0, pre1, w);
        }
    }
    mask();
    nf4_requant_round<false, kPortable>(s.bin, valid, w, packed, am);
}

// A call of two records (inline): a restore fused with the next perturbation,
// or an update of two records, where the per-tile work around the noise weighs
// most (one-record calls run engine_nf4_sweep_kernel). A whole tile (every
// tile but a tensor's last) takes a path compiled without bounds or masks, its
// codes and absmax addressed as the tile's scalar base plus a 32-bit lane
// offset; the 8 lanes of a block all store its absmax (the same value to the
// same address). With no records (out of place with nothing to apply) a tile
// is copied. NF4 tensors are never shards (first = 0), so element e of the
// tile is element e of the tensor. Compiled for 8 waves per SIMD (at most 64
// VGPRs), the occupancy of the other kernels.
template <bool kPortable>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(kPortable ? 1 : 8, 8)))
void engine_nf4_short_kernel(EngineArgs a)
{
    const uint32_t tile = blockIdx.x;  // the grid is exactly the tiles of this table (< 2^31)
    const uint32_t ti = a.tile_tensor[tile];
    const TensorDesc d = a.tensors[ti];
    __shared__ NF4ShortLds lds;
    // out of place: read tensor ti of the source set (same layout), write d
    const uint64_t codes = a.src_tensors ? a.src_tensors[ti].data : d.data;
    const uint64_t absmax = a.src_tensors ? a.src_tensors[ti].aux : d.aux;
    const uint32_t local = tile - uint32_t(d.tile_begin);
    const uint32_t lane = threadIdx.x;
    if (local < uint32_t(d.numel / kTileNF4)) {  // uniform: a whole tile
        constexpr uint32_t kWords = kTileNF4 / 8, kBlocks = kTileNF4 / kNF4Block;  // per tile
        const MEZO_GLOBAL uint32_t* cin = reinterpret_cast<const MEZO_GLOBAL uint32_t*>(codes) + uint64_t(local) * kWords;
        const gfloat_t* ain = reinterpret_cast<const gfloat_t*>(absmax) + uint64_t(local) * kBlocks;
        uint32_t packed = __builtin_nontemporal_load(cin + lane);
        float am = ain[lane >> 3];
        nf4_short_lds_init(lds);
        if (a.n_rec) short_records<kPortable, true>(a, d.tensor_id, local * uint32_t(kTileNF4 / 4) + 2 * lane, 0xFFu,
                                                    lds, packed, am);
        MEZO_GLOBAL uint32_t* cout = reinterpret_cast<MEZO_GLOBAL uint32_t*>(d.data) + uint64_t(local) * kWords;
        gfloat_t* aout = reinterpret_cast<gfloat_t*>(d.aux) + uint64_t(local) * kBlocks;
        __builtin_nontemporal_store(packed, cout + lane);
        aout[lane >> 3] = am;
    } else {
        const uint64_t e0 = uint64_t(local) * kTileNF4 + lane * 8u;
        uint32_t packed;
        float am;
        nf4_load(codes, absmax, e0, d.numel, packed, am);
        nf4_short_lds_init(lds);
        if (a.n_rec)
            short_records<kPortable, false>(a, d.tensor_id, uint32_t(e0 >> 2), nf4_valid(e0, d.numel), lds, packed,
                                            am);
        nf4_store(d.data, d.aux, e0, d.numel, packed, am);
    }
}

// Block maxima and coefficients for which the fast sweep works on w / am
// (below): am in [2^-64, 2^64] and |c| <= 2^60, so that c / am, the values
// v + (c / am) z and am times their maximum stay finite.
constexpr uint32_t kFoldAmLo = 0x1F800000u;  // 2^-64
constexpr uint32_t kFoldAmHi = 0x5F800000u;  // 2^64
constexpr float kFoldCoefMax = 0x1p60f;

// A lane's 16 elements (Philox blocks blk .. blk + 3 of its tensor) through a
// call of one record: dequantize, add the noise (fast mode: straight into the
// values, as short_step; portable mode: acc = c z, then w + acc), quantize.
// Fast mode, when every lane's block maximum am and the coefficient c are in
// range (uniform): the values are kept divided by am, v + (c / am) z with v
// the table values themselves, and the new absmax is am times their maximum.
// The quantizer only sees the ratio w / max |w|, so codes and absmax are those
// of v am + c z up to a few roundings (within the fast mode's tolerance), and
// the 16 products v am are saved. Otherwise the values are v am as in
// portable mode.
template <bool kPortable, bool kFull>
__device__ __forceinline__ void sweep16(const SeedRec& rec, uint32_t tensor_id, uint32_t blk, uint32_t valid,
                                        const NF4ShortLds& s, uint32_t (&packed)[2], float& am)
{
    float w[16];
    float c = rec.coef;
    float scale = 1.0f;  // the factor from the quantized values' maximum to the new absmax
    if constexpr (kPortable) {
        nf4_dequant_pairs16(s, packed, am, valid, w);
    } else {
        const bool in_range = __float_as_uint(am) - kFoldAmLo <= kFoldAmHi - kFoldAmLo;
        if (__builtin_amdgcn_ballot_w64(!in_range) == 0 && fabsf(c) <= kFoldCoefMax) {  // uniform
            nf4_dequant_pairs16(s, packed, 1.0f, valid, w);
            c = c * __builtin_amdgcn_rcpf(am);
            scale = am;
        } else {
            nf4_dequant_pairs16(s, packed, am, valid, w);
        }
    }
    const SeedUniform u = seed_uniform(rec, tensor_id);
#pragma unroll
    for (int h = 0; h < 4; ++h) {
        uint32_t w0, w1, w2, w3;
        philox_words(u, block_pre(blk + h), w0, w1, w2, w3);
        float* w4 = w + 4 * h;
        if constexpr (kPortable) {
            const Z4 z = gauss4_portable(w0, w1, w2, w3);
            w4[0] = w4[0] + rec.coef * z.z0;
            w4[1] = w4[1] + rec.coef * z.z1;
            w4[2] = w4[2] + rec.coef * z.z2;
            w4[3] = w4[3] + rec.coef * z.z3;
        } else {
            box_muller_pair_acc(w0, w1, c, w4[0], w4[1]);
            box_muller_pair_acc(w2, w3, c, w4[2], w4[3]);
        }
    }
    if (!kFull && partial_wave16(valid)) {  // only waves that reach a tensor's end
#pragma unroll
        for (int j = 0; j < 16; ++j)
            if (!((valid >> j) & 1u)) w[j] = 0.0f;
    }
    nf4_requant_round16<kPortable>(s.bin, valid, w, packed, am);
    if constexpr (!kPortable) am = am * scale;
}

// A call of one record (a perturbation): 16 elements per lane, 128-lane
// workgroups over the same 2048-element tiles (nf4_ops.hpp). Whole tiles are
// addressed as in engine_nf4_short_kernel (codes: 8 bytes per lane; absmax
// stored by the block's 4 lanes); the last tile of a tensor reads and writes
// its code bytes one by one.
template <bool kPortable>
__global__ __launch_bounds__(kSweepLanes) __attribute__((amdgpu_waves_per_eu(8, 8)))
void engine_nf4_sweep_kernel(EngineArgs a)
{
    const uint32_t tile = blockIdx.x;  // the grid is exactly the tiles of this table (< 2^31)
    const uint32_t ti = a.tile_tensor[tile];
    const TensorDesc d = a.tensors[ti];
    __shared__ NF4ShortLds lds;
    // out of place: read tensor ti of the source set (same layout), write d
    const uint64_t codes = a.src_tensors ? a.src_tensors[ti].data : d.data;
    const uint64_t absmax = a.src_tensors ? a.src_tensors[ti].aux : d.aux;
    const uint32_t local = tile - uint32_t(d.tile_begin);
    const uint32_t lane = threadIdx.x;
    if (local < uint32_t(d.numel / kTileNF4)) {  // uniform: a whole tile
        constexpr uint32_t kPairs = kTileNF4 / 16, kBlocks = kTileNF4 / kNF4Block;  // per tile
        const gu32x2_t* cin = reinterpret_cast<const gu32x2_t*>(codes) + uint64_t(local) * kPairs;
        const gfloat_t* ain = reinterpret_cast<const gfloat_t*>(absmax) + uint64_t(local) * kBlocks;
        const u32x2_t v = __builtin_nontemporal_load(cin + lane);
        uint32_t packed[2] = {v.x, v.y};
        float am = ain[lane >> 2];
        nf4_sweep_lds_init(lds);
        sweep16<kPortable, true>(a.inl[0], d.tensor_id, local * uint32_t(kTileNF4 / 4) + 4 * lane, 0xFFFFu, lds,
                                 packed, am);
        gu32x2_t* cout = reinterpret_cast<gu32x2_t*>(d.data) + uint64_t(local) * kPairs;
        gfloat_t* aout = reinterpret_cast<gfloat_t*>(d.aux) + uint64_t(local) * kBlocks;
        const u32x2_t o = {packed[0], packed[1]};
        __builtin_nontemporal_store(o, cout + lane);
        aout[lane >> 2] = am;
    } else {
        const uint64_t e0 = uint64_t(local) * kTileNF4 + lane * 16u;
        uint32_t packed[2] = {0u, 0u};
        float am = 0.0f;
        if (e0 < d.numel) {
            const MEZO_GLOBAL uint8_t* cb = reinterpret_cast<const MEZO_GLOBAL uint8_t*>(codes + e0 / 2);
#pragma unroll
            for (uint32_t k = 0; k < 8; ++k)
                if (e0 + 2 * k < d.numel) packed[k >> 2] |= uint32_t(cb[k]) << (8 * (k & 3));
            am = reinterpret_cast<const gfloat_t*>(absmax)[e0 / kNF4Block];
        }
        nf4_sweep_lds_init(lds);
        sweep16<kPortable, false>(a.inl[0], d.tensor_id, uint32_t(e0 >> 2), nf4_valid16(e0, d.numel), lds, packed,
                                  am);
        if (e0 < d.numel) {
            MEZO_GLOBAL uint8_t* ob = reinterpret_cast<MEZO_GLOBAL uint8_t*>(d.data + e0 / 2);
#pragma unroll
            for (uint32_t k = 0; k < 8; ++k)
                if (e0 + 2 * k < d.numel) ob[k] = uint8_t(packed[k >> 2] >> (8 * (k & 3)));
            reinterpret_cast<gfloat_t*>(d.aux)[e0 / kNF4Block] = am;
        }
    }
}

// Record lists of more than two records: one loop over the records (tile_nf4).
template <bool kInline, bool kPortable>
__global__ __launch_bounds__(kThreads) void engine_nf4_kernel(EngineArgs a)
{
    const uint64_t tile = blockIdx.x;  // the grid is exactly the tiles of this table
    const uint32_t ti = a.tile_tensor[tile];
    const TensorDesc d = a.tensors[ti];
    __shared__ NF4Lds lds;
    // out of place: read tensor ti of the source set (same layout), write d
    const uint64_t codes = a.src_tensors ? a.src_tensors[ti].data : d.data;
    const uint64_t absmax = a.src_tensors ? a.src_tensors[ti].aux : d.aux;
    const uint64_t local = tile - d.tile_begin;
    const uint64_t e0 = local * kTileNF4 + threadIdx.x * 8u;
    uint32_t packed;
    float am;
    nf4_load(codes, absmax, e0, d.numel, packed, am);
    nf4_lds_init(lds);
    tile_nf4<kInline, kPortable, false>(a, d, e0, packed, am, lds);
}

namespace {
hipError_t launch1(void (*kernel)(EngineArgs), dim3 g, dim3 b, hipStream_t stream, EngineArgs arg)
{
    void* params[] = {&arg};
    return hipLaunchKernel(reinterpret_cast<const void*>(kernel), g, b, params, 0, stream);
}

template <bool kPortable>
hipError_t launch_variant(const EngineArgs& args, dim3 g, dim3 b, hipStream_t stream)
{
    if (args.n_rec > kInlineRecs) return launch1(engine_nf4_kernel<false, kPortable>, g, b, stream, args);
    if (args.n_rec == 1)
        return launch1(engine_nf4_sweep_kernel<kPortable>, g, dim3{uint32_t(kSweepLanes)}, stream, args);
    if (args.n_rec <= 2) return launch1(engine_nf4_short_kernel<kPortable>, g, b, stream, args);
    return launch1(engine_nf4_kernel<true, kPortable>, g, b, stream, args);
}
}  // namespace

hipError_t launch_engine_nf4(const EngineArgs& args, bool portable, hipStream_t stream)
{
    if (args.total_tiles == 0) return hipSuccess;
    if (args.total_tiles > uint64_t(0x7FFFFFFF)) return hipErrorInvalidValue;
    const dim3 g{uint32_t(args.total_tiles)};
    const dim3 b{uint32_t(kThreads)};
    return portable ? launch_variant<true>(args, g, b, stream) : launch_variant<false>(args, g, b, stream);
}

}  // namespace mezo
