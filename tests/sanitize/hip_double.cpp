// hip_double.cpp — TEST INFRASTRUCTURE ONLY: a host-memory stand-in for the
// HIP runtime calls and the kernel launchers that the C ABI's host code
// (api.cpp) makes, so that api.cpp can be built with AddressSanitizer and
// UndefinedBehaviorSanitizer and driven on a machine without a GPU.
//
// "Device" memory is host memory from malloc, tracked by address and size;
// events are heap objects; streams are opaque tokens. A "launch" runs no
// kernel: it reads every byte the real kernel would read from the library's
// own device tables and staged record lists (so a bookkeeping mistake there is
// an out-of-bounds or use-after-free read the sanitizer reports), checks that
// they describe a consistent launch, and records what was launched for the
// driver (abi_host_check.c) to inspect through the double_* functions.
#include <hip/hip_runtime_api.h>

#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <vector>

#include "checksum_launch.hpp"
#include "engine_launch.hpp"
#include "inspect.hpp"
#include "nf4_launch.hpp"
#include "noalloc_launch.hpp"
#include "records.hpp"

namespace {

std::mutex g_mu;
std::map<uintptr_t, size_t> g_dev;   // live "device" allocations: address -> bytes
std::map<uintptr_t, size_t> g_host;  // live pinned host allocations
int g_device = 0;
int g_capturing = 0;
long g_fail_malloc_in = -1;          // fail the n-th hipMalloc from now (0 = the next)

struct Stats {
    unsigned long launches[3];       // engine launches per storage type
    unsigned long checksum_launches;
    unsigned long nf4_launches;
    unsigned long generate_launches;
    unsigned long event_syncs;
    unsigned long events_live;
    unsigned long h2d_bytes;
    unsigned long allocations;       // hipMalloc + hipHostMalloc + hipEventCreateWithFlags calls
    unsigned long stage_launches;
} g_stats;

// the file-scope staging array of the entry point that allocates nothing
mezo::SeedRec g_scratch[mezo::kNoAllocRecords];

std::vector<mezo::SeedRec> g_last_recs;
uint32_t g_last_dtype = 0;
int g_last_out_of_place = 0;

struct Event {
    uint32_t magic;
    int recorded;
};
constexpr uint32_t kEventMagic = 0x45564E54u;

[[noreturn]] void fail(const char* what)
{
    std::fprintf(stderr, "hip_double: %s\n", what);
    std::abort();
}

// [p, p + bytes) lies inside one live allocation of the map.
bool inside(const std::map<uintptr_t, size_t>& m, const void* p, size_t bytes)
{
    const uintptr_t a = reinterpret_cast<uintptr_t>(p);
    auto it = m.upper_bound(a);
    if (it == m.begin()) return false;
    --it;
    return a >= it->first && a + bytes <= it->first + it->second;
}

// Read every byte of [p, p + bytes) (the sanitizer checks each access).
uint64_t touch(const void* p, size_t bytes)
{
    const volatile unsigned char* c = static_cast<const volatile unsigned char*>(p);
    uint64_t s = 0;
    for (size_t i = 0; i < bytes; ++i) s += c[i];
    return s;
}

void check_table(const mezo::TensorDesc* t, uint32_t n, const uint32_t* tile_tensor, uint64_t tiles)
{
    if (!inside(g_dev, t, n * sizeof(mezo::TensorDesc))) fail("tensor table is not a live device allocation");
    if (!inside(g_dev, tile_tensor, tiles * sizeof(uint32_t))) fail("tile map is not a live device allocation");
    touch(t, n * sizeof(mezo::TensorDesc));
    for (uint64_t tile = 0; tile < tiles; ++tile) {
        const uint32_t i = tile_tensor[tile];
        if (i >= n) fail("tile map names a tensor past the table");
        const uint64_t end = i + 1 < n ? t[i + 1].tile_begin : tiles;
        if (tile < t[i].tile_begin || tile >= end) fail("tile map and tensor table disagree");
    }
}

}  // namespace

// ---- the HIP runtime calls api.cpp makes -------------------------------------

extern "C" {

const char* hipGetErrorString(hipError_t e) { return e == hipSuccess ? "no error" : "hip_double error"; }

hipError_t hipGetDevice(int* d)
{
    *d = g_device;
    return hipSuccess;
}

hipError_t hipMalloc(void** p, size_t bytes)
{
    std::lock_guard<std::mutex> lock(g_mu);
    if (g_fail_malloc_in == 0) {
        g_fail_malloc_in = -1;
        *p = nullptr;
        return hipErrorOutOfMemory;
    }
    if (g_fail_malloc_in > 0) --g_fail_malloc_in;
    ++g_stats.allocations;
    *p = std::malloc(bytes ? bytes : 1);
    if (!*p) return hipErrorOutOfMemory;
    g_dev[reinterpret_cast<uintptr_t>(*p)] = bytes;
    return hipSuccess;
}

hipError_t hipFree(void* p)
{
    std::lock_guard<std::mutex> lock(g_mu);
    if (!p) return hipSuccess;
    if (!g_dev.erase(reinterpret_cast<uintptr_t>(p))) fail("hipFree of an address hipMalloc did not return");
    std::free(p);
    return hipSuccess;
}

hipError_t hipHostMalloc(void** p, size_t bytes, unsigned int)
{
    std::lock_guard<std::mutex> lock(g_mu);
    ++g_stats.allocations;
    *p = std::malloc(bytes ? bytes : 1);
    if (!*p) return hipErrorOutOfMemory;
    g_host[reinterpret_cast<uintptr_t>(*p)] = bytes;
    return hipSuccess;
}

hipError_t hipHostFree(void* p)
{
    std::lock_guard<std::mutex> lock(g_mu);
    if (!p) return hipSuccess;
    if (!g_host.erase(reinterpret_cast<uintptr_t>(p))) fail("hipHostFree of an address hipHostMalloc did not return");
    std::free(p);
    return hipSuccess;
}

hipError_t hipMemcpy(void* dst, const void* src, size_t bytes, hipMemcpyKind kind)
{
    std::lock_guard<std::mutex> lock(g_mu);
    if (kind != hipMemcpyHostToDevice) fail("unexpected copy direction");
    if (!inside(g_dev, dst, bytes)) fail("hipMemcpy past a device allocation");
    std::memcpy(dst, src, bytes);
    g_stats.h2d_bytes += bytes;
    return hipSuccess;
}

hipError_t hipMemcpyAsync(void* dst, const void* src, size_t bytes, hipMemcpyKind kind, hipStream_t)
{
    std::lock_guard<std::mutex> lock(g_mu);
    if (kind != hipMemcpyHostToDevice) fail("unexpected copy direction");
    if (!inside(g_dev, dst, bytes)) fail("hipMemcpyAsync past a device allocation");
    if (!inside(g_host, src, bytes)) fail("hipMemcpyAsync from outside a pinned host allocation");
    std::memcpy(dst, src, bytes);
    g_stats.h2d_bytes += bytes;
    return hipSuccess;
}

hipError_t hipStreamIsCapturing(hipStream_t, hipStreamCaptureStatus* st)
{
    *st = g_capturing ? hipStreamCaptureStatusActive : hipStreamCaptureStatusNone;
    return hipSuccess;
}

hipError_t hipEventCreateWithFlags(hipEvent_t* e, unsigned)
{
    Event* ev = new Event{kEventMagic, 0};
    *e = reinterpret_cast<hipEvent_t>(ev);
    std::lock_guard<std::mutex> lock(g_mu);
    ++g_stats.events_live;
    ++g_stats.allocations;
    return hipSuccess;
}

hipError_t hipEventRecord(hipEvent_t e, hipStream_t)
{
    Event* ev = reinterpret_cast<Event*>(e);
    if (!ev || ev->magic != kEventMagic) fail("hipEventRecord on a destroyed or foreign event");
    ev->recorded = 1;
    return hipSuccess;
}

hipError_t hipEventSynchronize(hipEvent_t e)
{
    Event* ev = reinterpret_cast<Event*>(e);
    if (!ev || ev->magic != kEventMagic) fail("hipEventSynchronize on a destroyed or foreign event");
    std::lock_guard<std::mutex> lock(g_mu);
    ++g_stats.event_syncs;
    return hipSuccess;
}

hipError_t hipEventDestroy(hipEvent_t e)
{
    Event* ev = reinterpret_cast<Event*>(e);
    if (!ev || ev->magic != kEventMagic) fail("hipEventDestroy of a destroyed or foreign event");
    ev->magic = 0;
    delete ev;
    std::lock_guard<std::mutex> lock(g_mu);
    --g_stats.events_live;
    return hipSuccess;
}

}  // extern "C"

// ---- the kernel launchers ------------------------------------------------------

namespace mezo {

namespace {
hipError_t engine(const EngineArgs& a, uint32_t dtype)
{
    std::lock_guard<std::mutex> lock(g_mu);
    check_table(a.tensors, a.n_tensors, a.tile_tensor, a.total_tiles);
    for (uint32_t i = 0; i < a.n_tensors; ++i)
        if (a.tensors[i].dtype != dtype) fail("a launch mixes storage types");
    if (a.src_tensors) {
        if (!inside(g_dev, a.src_tensors, a.n_tensors * sizeof(TensorDesc))) fail("source table is not live");
        touch(a.src_tensors, a.n_tensors * sizeof(TensorDesc));
    }
    const SeedRec* recs = a.inl;
    if (a.n_rec > kInlineRecs) {
        if (!inside(g_dev, a.ext, size_t(a.n_rec) * sizeof(SeedRec))) fail("staged records past their buffer");
        recs = a.ext;
    }
    touch(recs, size_t(a.n_rec) * sizeof(SeedRec));
    if (a.n_rec > 0 && recs[a.n_rec - 1].last != 1u) fail("a launch's last record does not end a step");
    if (a.n_rec == 0 && !a.src_tensors) fail("an in-place launch without records");
    g_last_recs.assign(recs, recs + a.n_rec);
    g_last_dtype = dtype;
    g_last_out_of_place = a.src_tensors != nullptr;
    ++g_stats.launches[dtype];
    return hipSuccess;
}
}  // namespace

hipError_t launch_engine_dense(const EngineArgs& a, uint32_t dtype, bool, hipStream_t)
{
    if (dtype != kF32 && dtype != kBF16) fail("dense launch of another storage type");
    return engine(a, dtype);
}

hipError_t launch_engine_nf4(const EngineArgs& a, bool, hipStream_t) { return engine(a, kNF4); }

hipError_t launch_checksum(const ChecksumArgs* tables, const uint32_t* dtypes, int n, unsigned long long* out,
                           unsigned long long* acc, int, hipStream_t)
{
    std::lock_guard<std::mutex> lock(g_mu);
    // the running sum: two words of a device allocation, zero between calls
    if (!inside(g_dev, acc, 2 * sizeof(*acc))) fail("checksum running sum outside a device allocation");
    if (acc[0] != 0 || acc[1] != 0) fail("checksum running sum not zero at a call");
    (void)out;
    for (int i = 0; i < n; ++i) {
        const TensorDesc* t = tables[i].tensors;
        uint32_t cnt = 0;
        // the table's length is not passed: count the entries that the tile
        // map names
        for (uint64_t tile = 0; tile < tables[i].total_tiles; ++tile) {
            if (!inside(g_dev, tables[i].tile_tensor + tile, 4)) fail("checksum tile map past its buffer");
            cnt = tables[i].tile_tensor[tile] + 1 > cnt ? tables[i].tile_tensor[tile] + 1 : cnt;
        }
        check_table(t, cnt, tables[i].tile_tensor, tables[i].total_tiles);
        for (uint32_t k = 0; k < cnt; ++k)
            if (t[k].dtype != dtypes[i]) fail("checksum table of mixed storage types");
    }
    ++g_stats.checksum_launches;
    return hipSuccess;
}

hipError_t noalloc_scratch(SeedRec** out)
{
    std::lock_guard<std::mutex> lock(g_mu);
    // registered as device memory so that the engine launch may read it
    g_dev[reinterpret_cast<uintptr_t>(g_scratch)] = sizeof(g_scratch);
    *out = g_scratch;
    return hipSuccess;
}

hipError_t launch_stage(SeedRec* dst, uint32_t offset, const SeedRec* recs, uint32_t n, hipStream_t)
{
    if (dst != g_scratch) fail("staging outside the staging array");
    if (n == 0 || n > kStageRecs || offset > kNoAllocRecords - n) fail("staging past the staging array");
    std::lock_guard<std::mutex> lock(g_mu);
    std::memcpy(dst + offset, recs, n * sizeof(SeedRec));
    ++g_stats.stage_launches;
    return hipSuccess;
}

hipError_t launch_nf4(const NF4ConvArgs& a, bool, hipStream_t)
{
    if (a.n == 0 || (a.dtype != kF32 && a.dtype != kBF16)) fail("bad NF4 conversion");
    std::lock_guard<std::mutex> lock(g_mu);
    ++g_stats.nf4_launches;
    return hipSuccess;
}

hipError_t launch_generate(const GenArgs& a, hipStream_t)
{
    if (a.count == 0) fail("empty generate launch");
    std::lock_guard<std::mutex> lock(g_mu);
    ++g_stats.generate_launches;
    return hipSuccess;
}

hipError_t launch_box_muller(const uint32_t*, uint64_t n_blocks, uint32_t, float*, hipStream_t)
{
    if (n_blocks == 0) fail("empty transform launch");
    std::lock_guard<std::mutex> lock(g_mu);
    ++g_stats.generate_launches;
    return hipSuccess;
}

}  // namespace mezo

// ---- control and inspection for the driver ----------------------------------

extern "C" {

void double_set_device(int d) { g_device = d; }
void double_set_capturing(int on) { g_capturing = on; }
void double_fail_malloc_in(long n) { g_fail_malloc_in = n; }

unsigned long double_engine_launches(uint32_t dtype) { return g_stats.launches[dtype]; }
unsigned long double_checksum_launches(void) { return g_stats.checksum_launches; }
unsigned long double_nf4_launches(void) { return g_stats.nf4_launches; }
unsigned long double_generate_launches(void) { return g_stats.generate_launches; }
unsigned long double_event_syncs(void) { return g_stats.event_syncs; }
unsigned long double_events_live(void) { return g_stats.events_live; }
size_t double_device_allocations(void)
{
    return g_dev.size() + g_host.size() - g_dev.count(reinterpret_cast<uintptr_t>(g_scratch));
}
unsigned long double_allocation_calls(void) { return g_stats.allocations; }
unsigned long double_stage_launches(void) { return g_stats.stage_launches; }

// The records of the last engine launch: their count, and for each its
// coefficient, step-end flag and low machine word (arrays of at least max).
uint32_t double_last_records(float* coef, uint32_t* last, uint32_t* machine, uint32_t max)
{
    const uint32_t n = static_cast<uint32_t>(g_last_recs.size());
    for (uint32_t i = 0; i < n && i < max; ++i) {
        coef[i] = g_last_recs[i].coef;
        last[i] = g_last_recs[i].last;
        machine[i] = g_last_recs[i].key0;
    }
    return n;
}

int double_last_out_of_place(void) { return g_last_out_of_place; }

}  // extern "C"
