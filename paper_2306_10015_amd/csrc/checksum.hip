// checksum.hip — the 64-bit checksum of theta (ChecksumMatch, Algorithm 1):
// a read-only stream over the same tiles as the engine; every lane sums the
// mixes of its 8-byte chunks, a workgroup reduces across lanes and waves and
// adds its sum to a running sum with one 64-bit atomic, and the last
// workgroup of the call writes the total out. Sums mod 2^64 commute, so the
// grid shape and the order of the atomics do not change the result.
#include <atomic>

#include "checksum_launch.hpp"
#include "stream_io.hpp"
#include "tiles.hpp"

namespace mezo {

__device__ __forceinline__ uint64_t fmix64(uint64_t x)
{
    x ^= x >> 33;
    x *= kFmixA;
    x ^= x >> 33;
    x *= kFmixB;
    x ^= x >> 33;
    return x;
}

// Reduce every lane's sum across the workgroup and add it to the running sum
// a.acc[0] with one 64-bit atomic; then take a ticket (a.acc[1]). The
// workgroup that takes the launch's last ticket finds every other one's sum
// in acc[0]; it clears the ticket for the next launch and, at the call's last
// launch, moves the total to *out and clears the sum: no launch has to zero
// anything first. Ordering without cache maintenance: the add returns the old
// sum and the wave waits for that value (the add has then been performed
// where all atomics on acc are) before it takes its ticket, so every sum
// precedes its ticket, and the last ticket's holder reads acc[0] by an atomic
// too. (A device-scope fence here, an L2 write-back and invalidate in every
// workgroup, made the 125M fp32 checksum kernel 20% slower.) All lanes of the
// workgroup must call it.
__device__ __forceinline__ void add_workgroup_sum(uint64_t sum, const ChecksumArgs& a)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) sum += __shfl_xor(sum, off);
    __shared__ uint64_t part[kThreads / 64];
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = sum;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint64_t s = 0;
#pragma unroll
        for (int i = 0; i < kThreads / 64; ++i) s += part[i];
        unsigned long long old = atomicAdd(a.acc, static_cast<unsigned long long>(s));
        asm volatile("" : "+v"(old) : : "memory");  // the returned value is waited for here
        if (atomicAdd(a.acc + 1, 1ull) == gridDim.x - 1ull) {
            if (a.last) *a.out = atomicExch(a.acc, 0ull);
            atomicExch(a.acc + 1, 0ull);
        }
    }
}

// A lane's 16 bytes of a tile that lies wholly inside its tensor: the
// tile's base plus a 32-bit lane offset, no bounds.
__device__ __forceinline__ u32x4_t load_whole_tile(uint64_t data, uint64_t local)
{
    const gu32x4_t* base = reinterpret_cast<const gu32x4_t*>(data) + local * kThreads;
    return __builtin_nontemporal_load(base + threadIdx.x);
}

// The mixes of a lane's two chunks of a whole tile: chunk numbers as the
// tile's uniform part plus the lane's constant part.
__device__ __forceinline__ uint64_t mix_whole_tile(u32x4_t v, uint64_t cpos_tile, uint64_t tmix, uint64_t cpos_lane)
{
    const uint64_t p0 = cpos_tile + cpos_lane;  // (its first chunk's number) * kChunkPos
    const uint64_t lo = uint64_t(v.x) | (uint64_t(v.y) << 32);
    const uint64_t hi = uint64_t(v.z) | (uint64_t(v.w) << 32);
    return fmix64(lo ^ p0 ^ tmix) + fmix64(hi ^ (p0 + kChunkPos) ^ tmix);
}

// A lane's share of a tensor's last tile, which the tensor's end may cut:
// only the elements that exist, the last chunk zero-padded.
template <uint32_t kDtype>
__device__ __forceinline__ uint64_t mix_last_tile(const TensorDesc& d, uint64_t local)
{
    constexpr uint64_t kPer = Layout<kDtype>::kPerGroup;
    constexpr uint64_t kEsz = 16 / kPer;
    const uint64_t nchunks = (d.numel * kEsz + 7) / 8;
    const uint64_t cbase = d.first * kEsz / 8;  // chunk number of the shard's first byte
    const uint64_t tmix = uint64_t(d.tensor_id) * kChunkTensor;
    const uint64_t grp = group_index<1>(local, 0);
    const uint64_t c0 = grp * 2;  // the group's first chunk within the shard
    if (c0 >= nchunks) return 0;
    uint4 v;
    if ((grp + 1) * kPer <= d.numel) {
        v = load_stream(d.data + grp * 16);
    } else {
        uint32_t w[4] = {0u, 0u, 0u, 0u};
        if constexpr (kDtype == kF32) {
            const MEZO_GLOBAL uint32_t* in = reinterpret_cast<const MEZO_GLOBAL uint32_t*>(d.data);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (grp * 4 + j < d.numel) w[j] = in[grp * 4 + j];
        } else {
            const gu16_t* in = reinterpret_cast<const gu16_t*>(d.data);
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (grp * 8 + j < d.numel) w[j >> 1] |= uint32_t(in[grp * 8 + j]) << (16 * (j & 1));
        }
        v = make_uint4(w[0], w[1], w[2], w[3]);
    }
    const uint64_t lo = uint64_t(v.x) | (uint64_t(v.y) << 32);
    const uint64_t hi = uint64_t(v.z) | (uint64_t(v.w) << 32);
    uint64_t s = fmix64(lo ^ ((cbase + c0) * kChunkPos) ^ tmix);
    if (c0 + 1 < nchunks) s += fmix64(hi ^ ((cbase + c0 + 1) * kChunkPos) ^ tmix);
    return s;
}

// The tensor a run of tiles is in: its descriptor's fields in scalar
// registers, moved forward tensor by tensor (the tensors of a table lie in
// tile order, each right after the one before).
template <uint64_t kTileElems>
struct RunCursor {
    const TensorDesc* tensors;
    uint32_t ti;
    uint64_t data, aux, numel, first, begin, end;  // end: one past the tensor's last tile
    uint32_t id;

    __device__ __forceinline__ void load(uint32_t i)
    {
        ti = i;
        data = tensors[i].data;
        aux = tensors[i].aux;
        numel = tensors[i].numel;
        first = tensors[i].first;
        begin = tensors[i].tile_begin;
        id = tensors[i].tensor_id;
        end = begin + (numel + kTileElems - 1) / kTileElems;
    }
    __device__ __forceinline__ void seek(uint64_t tile)
    {
        while (tile >= end) load(ti + 1);
    }
};

// fp32/bf16 tensors. Workgroup b takes the run of consecutive tiles
// [T b / G, T (b + 1) / G) of the table's T tiles (G workgroups, two per CU):
// the descriptor changes only where the run crosses into the next tensor (no
// per-tile map lookup). Tiles go in groups of eight where all lie wholly
// inside one tensor: the eight loads are issued before any is mixed, eight
// 16-byte loads in flight per lane. Few workgroups with many loads each
// stream faster than many with few: against eight workgroups per CU with
// two tiles in flight, the 125M fp32 set took 0.093 -> 0.085 ms and the 6.7B
// bf16 set 1.96 -> 1.90 ms (paired runs, checksums identical; one workgroup
// per CU or sixteen tiles in flight were slower).
template <uint32_t kDtype>
__global__ __launch_bounds__(kThreads) void checksum_kernel(ChecksumArgs a)
{
    static_assert(Layout<kDtype>::kGroups == 1, "one 16-byte group per lane");
    constexpr uint64_t kPer = Layout<kDtype>::kPerGroup;
    constexpr uint64_t kEsz = 16 / kPer;
    constexpr uint64_t kTileElems = uint64_t(kThreads) * kPer;
    constexpr uint64_t kInFlight = 8;  // tiles whose loads a lane issues before mixing any
    // chunk number of the lane's first chunk within its tile, times kChunkPos;
    // opaque from here on: otherwise the compiler folds uniform + lane
    // constant back into one per-lane 64-bit multiply in every tile
    uint64_t cpos_lane = 2 * uint64_t(threadIdx.x) * kChunkPos;
    asm("" : "+v"(cpos_lane));
    const uint64_t T = a.total_tiles;
    const uint64_t t0 = T * blockIdx.x / gridDim.x;
    const uint64_t t_end = T * (blockIdx.x + 1) / gridDim.x;
    uint64_t sum = 0;
    if (t0 < t_end) {
        RunCursor<kTileElems> c;
        c.tensors = a.tensors;
        c.load(a.tile_tensor[t0]);
        // the chunk-position term of tile `local` of the cursor's tensor
        const auto cpos_of = [&](uint64_t local) { return (c.first * kEsz / 8 + 2 * local * kThreads) * kChunkPos; };
        const auto one_tile = [&](uint64_t tile) {
            c.seek(tile);
            const uint64_t local = tile - c.begin;
            if ((local + 1) * kTileElems <= c.numel) {  // uniform: all but a tensor's last tile
                const u32x4_t v = load_whole_tile(c.data, local);
                sum += mix_whole_tile(v, cpos_of(local), uint64_t(c.id) * kChunkTensor, cpos_lane);
            } else {
                TensorDesc d;
                d.data = c.data;
                d.numel = c.numel;
                d.first = c.first;
                d.tensor_id = c.id;
                sum += mix_last_tile<kDtype>(d, local);
            }
        };
        uint64_t t = t0;
        for (; t + kInFlight <= t_end; t += kInFlight) {
            c.seek(t);
            const uint64_t local = t - c.begin;
            if ((local + kInFlight) * kTileElems <= c.numel) {  // uniform: all kInFlight tiles whole, one tensor
                u32x4_t v[kInFlight];
#pragma unroll
                for (uint64_t j = 0; j < kInFlight; ++j) v[j] = load_whole_tile(c.data, local + j);
                const uint64_t cpos = cpos_of(local);
                const uint64_t tmix = uint64_t(c.id) * kChunkTensor;
#pragma unroll
                for (uint64_t j = 0; j < kInFlight; ++j)
                    sum += mix_whole_tile(v[j], cpos + j * (2 * kThreads * kChunkPos), tmix, cpos_lane);
            } else {
                for (uint64_t j = 0; j < kInFlight; ++j) one_tile(t + j);
            }
        }
        for (; t < t_end; ++t) one_tile(t);
    }
    add_workgroup_sum(sum, a);
}

// A wave's share of an NF4 tensor's last tile, which the tensor's end may cut:
// the code chunks and absmax chunks that exist, the last of each zero-padded.
__device__ __forceinline__ uint64_t mix_nf4_last_tile(uint64_t data, uint64_t aux, uint64_t numel, uint64_t tmix,
                                                      uint64_t local, uint32_t lane)
{
    const uint64_t cbytes = (numel + 1) / 2;
    const uint64_t cchunks = (cbytes + 7) / 8;
    const uint64_t abytes = 4 * ((numel + kNF4Block - 1) / kNF4Block);
    uint64_t sum = 0;
    // codes: bytes [16u, 16u + 16) = chunks 2u, 2u + 1
    const uint64_t u = local * 64 + lane;
    if (16 * u < cbytes) {
        uint64_t lo = 0, hi = 0;
        if (16 * u + 16 <= cbytes) {
            const uint4 v = load_stream(data + 16 * u);
            lo = uint64_t(v.x) | (uint64_t(v.y) << 32);
            hi = uint64_t(v.z) | (uint64_t(v.w) << 32);
        } else {
            const MEZO_GLOBAL uint8_t* b = reinterpret_cast<const MEZO_GLOBAL uint8_t*>(data);
            for (uint64_t k = 16 * u; k < cbytes; ++k) {
                const uint64_t byte = uint64_t(b[k]);
                const uint64_t off = k - 16 * u;
                if (off < 8)
                    lo |= byte << (8 * off);
                else
                    hi |= byte << (8 * (off - 8));
            }
        }
        sum += fmix64(lo ^ (2 * u * kChunkPos) ^ tmix);
        if (16 * u + 8 < cbytes) sum += fmix64(hi ^ ((2 * u + 1) * kChunkPos) ^ tmix);
    }
    // absmax: bytes [ab, ab + 16) = absmax chunks k0, k0 + 1
    const uint64_t ab = local * (kTileNF4 / kNF4Block * 4) + 16 * uint64_t(lane);
    if (lane < kTileNF4 / kNF4Block * 4 / 16 && ab < abytes) {
        const uint64_t k0 = ab / 8;
        uint32_t f[4] = {0u, 0u, 0u, 0u};
        if (ab + 16 <= abytes) {
            const uint4 v = load_stream(aux + ab);
            f[0] = v.x;
            f[1] = v.y;
            f[2] = v.z;
            f[3] = v.w;
        } else {
            const MEZO_GLOBAL uint32_t* am = reinterpret_cast<const MEZO_GLOBAL uint32_t*>(aux);
            for (uint64_t k = ab; k < abytes; k += 4) f[(k - ab) / 4] = am[k / 4];
        }
        sum += fmix64((uint64_t(f[0]) | (uint64_t(f[1]) << 32)) ^ ((cchunks + k0) * kChunkPos) ^ tmix);
        if (ab + 8 < abytes)
            sum += fmix64((uint64_t(f[2]) | (uint64_t(f[3]) << 32)) ^ ((cchunks + k0 + 1) * kChunkPos) ^ tmix);
    }
    return sum;
}

// NF4 tensors: the code bytes zero-padded to whole chunks, then the absmax
// values, chunk numbers continuing. A tile of 2048 elements is one wave's:
// every lane reads 16 code bytes (two chunks) and lanes 0..15 a chunk of the
// tile's 128 absmax bytes. Wave w of W takes the run of consecutive tiles
// [T w / W, T (w + 1) / W), with its tensor's descriptor moved forward only
// where the run crosses into the next tensor, two whole tiles at a time.
__global__ __launch_bounds__(kThreads) void checksum_nf4_kernel(ChecksumArgs a)
{
    constexpr uint32_t kWaves = kThreads / 64;
    constexpr uint64_t kPair = 2;
    const uint32_t lane = threadIdx.x & 63u;
    // position terms of a lane's chunks within a tile, computed once (opaque
    // to the compiler, as in checksum_kernel): code chunks 2 lane, 2 lane + 1;
    // absmax chunk lane (lanes 0..15)
    uint64_t cpos_code = 2 * uint64_t(lane) * kChunkPos;
    uint64_t cpos_abs = uint64_t(lane & 15u) * kChunkPos;
    asm("" : "+v"(cpos_code));
    asm("" : "+v"(cpos_abs));
    const uint64_t W = uint64_t(gridDim.x) * kWaves;
    const uint64_t gw = uint64_t(blockIdx.x) * kWaves + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint64_t T = a.total_tiles;
    const uint64_t t0 = T * gw / W;
    const uint64_t t_end = T * (gw + 1) / W;
    uint64_t sum = 0;
    if (t0 < t_end) {
        RunCursor<kTileNF4> c;
        c.tensors = a.tensors;
        c.load(a.tile_tensor[t0]);
        // the mixes of whole tile `local` of the cursor's tensor from its
        // lane's code chunk v and absmax chunk f
        const auto mix_whole = [&](u32x4_t v, uint64_t f, uint64_t local) {
            const uint64_t tmix = uint64_t(c.id) * kChunkTensor;
            const uint64_t cchunks = ((c.numel + 1) / 2 + 7) / 8;
            const uint64_t p0 = 128 * local * kChunkPos + cpos_code;
            uint64_t s = fmix64((uint64_t(v.x) | (uint64_t(v.y) << 32)) ^ p0 ^ tmix);
            s += fmix64((uint64_t(v.z) | (uint64_t(v.w) << 32)) ^ (p0 + kChunkPos) ^ tmix);
            const uint64_t fm = fmix64(f ^ ((cchunks + 16 * local) * kChunkPos + cpos_abs) ^ tmix);
            return s + (lane < 16u ? fm : 0u);
        };
        // every lane loads absmax chunk (lane mod 16), so that both loads of a
        // tile issue before any mix
        const auto load_codes = [&](uint64_t local) {
            return __builtin_nontemporal_load(reinterpret_cast<const gu32x4_t*>(c.data) + local * 64 + lane);
        };
        const auto load_absmax = [&](uint64_t local) {
            return __builtin_nontemporal_load(reinterpret_cast<const MEZO_GLOBAL uint64_t*>(c.aux) + local * 16 +
                                              (lane & 15u));
        };
        const auto one_tile = [&](uint64_t tile) {
            c.seek(tile);
            const uint64_t local = tile - c.begin;
            if ((local + 1) * kTileNF4 <= c.numel) {  // uniform: a whole tile, 32 whole blocks
                const u32x4_t v = load_codes(local);
                const uint64_t f = load_absmax(local);
                sum += mix_whole(v, f, local);
            } else {
                sum += mix_nf4_last_tile(c.data, c.aux, c.numel, uint64_t(c.id) * kChunkTensor, local, lane);
            }
        };
        uint64_t t = t0;
        for (; t + kPair <= t_end; t += kPair) {
            c.seek(t);
            const uint64_t local = t - c.begin;
            if ((local + kPair) * kTileNF4 <= c.numel) {  // uniform: both tiles whole, one tensor
                u32x4_t v[kPair];
                uint64_t f[kPair];
#pragma unroll
                for (uint64_t j = 0; j < kPair; ++j) {
                    v[j] = load_codes(local + j);
                    f[j] = load_absmax(local + j);
                }
#pragma unroll
                for (uint64_t j = 0; j < kPair; ++j) sum += mix_whole(v[j], f[j], local + j);
            } else {
                for (uint64_t j = 0; j < kPair; ++j) one_tile(t + j);
            }
        }
        for (; t < t_end; ++t) one_tile(t);
    }
    add_workgroup_sum(sum, a);
}

__global__ void zero_u64_kernel(unsigned long long* out)
{
    if (threadIdx.x == 0 && blockIdx.x == 0) *out = 0ull;
}

namespace {
constexpr int kMaxDevices = 64;
std::atomic<int> g_cus[kMaxDevices];  // compute units per device, 0 = not yet asked

template <class Arg>
hipError_t launch1(void (*kernel)(Arg), dim3 g, dim3 b, hipStream_t stream, Arg arg)
{
    void* params[] = {&arg};
    return hipLaunchKernel(reinterpret_cast<const void*>(kernel), g, b, params, 0, stream);
}
}  // namespace

hipError_t launch_checksum(const ChecksumArgs* tables, const uint32_t* dtypes, int n_tables,
                           unsigned long long* out, unsigned long long* acc, int device, hipStream_t stream)
{
    if (device < 0 || device >= kMaxDevices) return hipErrorInvalidValue;
    int cus = g_cus[device].load(std::memory_order_relaxed);
    if (cus == 0) {
        hipError_t e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device);
        if (e != hipSuccess) return e;
        g_cus[device].store(cus, std::memory_order_relaxed);
    }
    int last = -1;  // the last table with tiles: its launch writes *out
    for (int i = 0; i < n_tables; ++i)
        if (tables[i].total_tiles) last = i;
    // no tiles at all (the C ABI never passes such a set): the checksum is 0
    if (last < 0) return launch1(zero_u64_kernel, dim3(1), dim3(64), stream, out);
    hipError_t e = hipSuccess;
    for (int i = 0; i <= last; ++i) {
        if (tables[i].total_tiles == 0) continue;
        ChecksumArgs args = tables[i];
        args.out = out;
        args.acc = acc;
        args.last = i == last ? 1u : 0u;
        // two workgroups per CU (NF4: four), each taking a run of
        // consecutive tiles (NF4: each of its waves a run of its own). NF4
        // with 8, 6, 4, 3, 2 per CU took 0.620, 0.614, 0.611, 0.640, 0.78 ms
        // on the 6.7B image (paired runs, checksums identical)
        const uint64_t per_wg = dtypes[i] == kNF4 ? kThreads / 64 : 1;
        const uint64_t need = (tables[i].total_tiles + per_wg - 1) / per_wg;
        const uint64_t cap = uint64_t(cus) * (dtypes[i] == kNF4 ? 4 : 2);
        const uint64_t grid = need < cap ? need : cap;
        const dim3 g{uint32_t(grid)};
        const dim3 b{uint32_t(kThreads)};
        if (dtypes[i] == kF32)
            e = launch1(checksum_kernel<kF32>, g, b, stream, args);
        else if (dtypes[i] == kBF16)
            e = launch1(checksum_kernel<kBF16>, g, b, stream, args);
        else
            e = launch1(checksum_nf4_kernel, g, b, stream, args);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace mezo
