// api.cpp — the C ABI of libmezo (include/mezo.h): argument checks, the
// paramset tensor table, the one-byte codec, seed records, staging and
// launches on the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <exception>
#include <memory>
#include <mutex>
#include <new>
#include <stdexcept>
#include <vector>

#include "../../include/mezo.h"
#include "checksum_launch.hpp"
#include "engine_launch.hpp"
#include "inspect.hpp"
#include "nf4_launch.hpp"
#include "noalloc_launch.hpp"
#include "records.hpp"

namespace {

// The last failure's message on this thread (a fixed buffer: reporting an
// error allocates nothing).
thread_local char t_last_error[256];

void set_error(const char* what, const char* detail = nullptr)
{
    std::snprintf(t_last_error, sizeof(t_last_error), detail ? "%s: %s" : "%s", what, detail);
}

int hip_fail(hipError_t e, const char* where)
{
    set_error(where, hipGetErrorString(e));
    return MEZO_EHIP;
}

// Runs the body of a C entry point: no C++ exception crosses the C ABI. The
// only ones the bodies can raise are host allocation failures (record lists,
// tables) and, in principle, a failing mutex.
template <class F>
int guarded(const char* what, F&& body) noexcept
{
    try {
        return body();
    } catch (const std::bad_alloc&) {
        set_error(what, "host allocation failed");
    } catch (const std::length_error&) {
        set_error(what, "host allocation failed");
    } catch (const std::exception& e) {
        set_error(what, e.what());
        return MEZO_EINVAL;
    } catch (...) {
        set_error(what, "unexpected exception");
        return MEZO_EINVAL;
    }
    return MEZO_ENOMEM;
}

#define MEZO_HIP(call)                                  \
    do {                                                \
        hipError_t err_ = (call);                       \
        if (err_ != hipSuccess) return hip_fail(err_, #call); \
    } while (0)

// ---- codec (Section 3: the projected gradient in one byte) -------------------

// Largest code magnitude: 127 (Section 3's clip), or for the signed log the
// largest k whose decoding fl32(exp(k / alpha) - 1) is finite when that is
// smaller (alpha < ~1.4314; the natural log, alpha = 1: 88).
int code_max(const mezo_codec_t& c)
{
    if (c.kind != MEZO_CODEC_SIGNED_LOG) return 127;
    int k = 127;
    while (k > 0 && !std::isfinite(static_cast<float>(std::expm1(double(k) / double(c.alpha))))) --k;
    return k;
}

bool codec_valid(const mezo_codec_t* c)
{
    if (!c) return false;
    if (c->kind == MEZO_CODEC_LINEAR) return std::isfinite(c->scale) && c->scale > 0.0f;
    if (c->kind == MEZO_CODEC_SIGNED_LOG)
        return std::isfinite(c->alpha) && c->alpha > 0.0f && code_max(*c) >= 1;
    return false;
}

int8_t encode(float g, const mezo_codec_t& c, double qmax)
{
    double r;
    if (c.kind == MEZO_CODEC_LINEAR) {
        r = double(std::rint(g / c.scale));  // fp32 quotient, ties to even
    } else {
        const double mag = std::rint(double(c.alpha) * std::log1p(std::fabs(double(g))));
        r = std::signbit(g) ? -mag : mag;
    }
    r = std::min(qmax, std::max(-qmax, r));
    return static_cast<int8_t>(r);
}

float decode(int8_t q, const mezo_codec_t& c)
{
    if (c.kind == MEZO_CODEC_LINEAR) return static_cast<float>(double(q) * double(c.scale));
    const double mag = std::expm1(std::fabs(double(q)) / double(c.alpha));
    return static_cast<float>(q < 0 ? -mag : mag);
}

// ---- seeds -----------------------------------------------------------------

bool seed_less(const mezo_seed_t& a, const mezo_seed_t& b)
{
    if (a.machine != b.machine) return a.machine < b.machine;
    if (a.step != b.step) return a.step < b.step;
    return a.sample < b.sample;
}

// fold: multiply the coefficient by the sqrt(2 ln 2) the fast kernels leave
// out of z (not for the portable Gaussian, whose kernels produce z itself).
mezo::SeedRec make_rec(const mezo_seed_t& s, float coef, bool last, bool fold)
{
    mezo::SeedRec r;
    r.key0 = static_cast<uint32_t>(s.machine);
    r.key1 = static_cast<uint32_t>(s.machine >> 32);
    r.step = s.step;
    const uint64_t p = uint64_t(mezo::kMulB) * uint64_t(s.sample);
    r.mb_hi = static_cast<uint32_t>(p >> 32);
    r.mb_lo = static_cast<uint32_t>(p);
    r.coef = fold ? static_cast<float>(double(coef) * mezo::kZScaleF64) : coef;
    r.last = last ? 1u : 0u;
    r.sample = s.sample;
    return r;
}

// Checks one step of the apply loop: the codec, lr, every code against the
// codec's range and the seeds strictly ascending (machine-timestamp order).
int check_step(const mezo_seed_t* seeds, const int8_t* q, uint32_t K, const mezo_codec_t* codec, float lr)
{
    if (!codec) return MEZO_EINVAL;
    if (!codec_valid(codec) || !std::isfinite(lr)) return MEZO_ERANGE;
    if (K == 0) return MEZO_OK;
    if (!seeds || !q) return MEZO_EINVAL;
    const int qmax = code_max(*codec);
    for (uint32_t k = 0; k < K; ++k)
        if (q[k] > qmax || q[k] < -qmax) return MEZO_ERANGE;  // -128 included
    for (uint32_t k = 1; k < K; ++k)
        if (!seed_less(seeds[k - 1], seeds[k])) return MEZO_EORDER;
    return MEZO_OK;
}

// Weight of perturbation k in the apply loop: -grad * lr (Algorithm 1).
float step_coef(int8_t q, const mezo_codec_t& codec, float lr)
{
    return static_cast<float>(-double(lr) * double(decode(q, codec)));
}

// Calls emit(record) for the records of a checked step in order: zero
// weights dropped, the step's last kept record flagged to round to storage.
// Returns how many it emitted.
template <class Emit>
uint32_t emit_step(const mezo_seed_t* seeds, const int8_t* q, uint32_t K, const mezo_codec_t& codec, float lr,
                   bool fold, Emit&& emit)
{
    uint32_t last = K;
    for (uint32_t k = K; k-- > 0;) {
        if (step_coef(q[k], codec, lr) != 0.0f) {
            last = k;
            break;
        }
    }
    uint32_t n = 0;
    for (uint32_t k = 0; last < K && k <= last; ++k) {
        const float c = step_coef(q[k], codec, lr);
        if (c == 0.0f) continue;
        emit(make_rec(seeds[k], c, k == last, fold));
        ++n;
    }
    return n;
}

// Checks one step of the apply loop and appends its records.
int append_step(const mezo_seed_t* seeds, const int8_t* q, uint32_t K, const mezo_codec_t* codec,
                float lr, bool fold, std::vector<mezo::SeedRec>& out)
{
    const int rc = check_step(seeds, q, K, codec, lr);
    if (rc || K == 0) return rc;
    emit_step(seeds, q, K, *codec, lr, fold, [&](const mezo::SeedRec& r) { out.push_back(r); });
    return MEZO_OK;
}

}  // namespace

// ---- paramset -----------------------------------------------------------------

struct mezo_paramset {
    static constexpr int kTypes = static_cast<int>(mezo::kStorageTypes);
    std::mutex mu;
    // One table per storage type (index = dtype), each in registration order
    // with tile_begin ascending; the engine runs one launch per non-empty table.
    std::vector<mezo::TensorDesc> table[kTypes];
    uint64_t total_tiles[kTypes] = {};
    uint64_t numel = 0;
    int device = -1;
    std::atomic<uint32_t> gaussian{MEZO_GAUSS_FAST};
    mezo::TensorDesc* d_table[kTypes] = {};
    uint32_t* d_tile_tensor[kTypes] = {};  // tensor index of every tile
    // One event per stream the paramset's kernels ran on, recorded after the
    // latest launch on that stream: destroy waits for all of them before it
    // frees the tables (work on an earlier stream may still be running). At
    // most kUses streams are tracked; a further stream takes over the entry
    // used longest ago, after waiting on the host for that entry's event. The
    // events are made with the device tables, at the first call, so that no
    // later call creates one.
    struct Use {
        hipStream_t stream = nullptr;
        hipEvent_t done = nullptr;
        uint64_t seq = 0;  // when the entry was last recorded; 0: not yet used
    };
    static constexpr size_t kUses = 16;
    Use uses[kUses];
    uint64_t use_seq = 0;
    // The checksum's running sums: two words per use entry (a stream's calls
    // are ordered, and an entry changes stream only after its work is done),
    // and one pair more for calls captured into a graph. Zero between calls.
    static constexpr size_t kCkPairs = kUses + 1;
    unsigned long long* d_ck = nullptr;

    // Staging of record lists too long for the kernel arguments: a ring of
    // slots, each reused only after the launch that read it has completed.
    struct Slot {
        mezo::SeedRec* host = nullptr;  // pinned
        mezo::SeedRec* dev = nullptr;
        size_t cap = 0;
        hipEvent_t done = nullptr;
    };
    static constexpr int kSlots = 4;
    Slot slots[kSlots];
    unsigned next_slot = 0;
};

namespace {

// The Gaussian a call uses, read once per call: its records are made for it
// (the fast kernels take the coefficient with sqrt(2 ln 2) folded in) and its
// launches run it, even if mezo_paramset_set_gaussian runs meanwhile.
bool portable_of(const mezo_paramset* ps) { return ps->gaussian.load() == MEZO_GAUSS_PORTABLE; }

// Device resources are made on first use, on the device current then.
int ensure_device(mezo_paramset* ps)
{
    int dev = -1;
    MEZO_HIP(hipGetDevice(&dev));
    if (ps->device >= 0) {
        if (dev != ps->device) {
            set_error("paramset used on a device other than the one it was first used on");
            return MEZO_EINVAL;
        }
        return MEZO_OK;
    }
    hipError_t e = hipSuccess;
    for (int dt = 0; dt < mezo_paramset::kTypes && e == hipSuccess; ++dt) {
        const std::vector<mezo::TensorDesc>& tab = ps->table[dt];
        if (tab.empty()) continue;
        const size_t bytes = tab.size() * sizeof(mezo::TensorDesc);
        e = hipMalloc(reinterpret_cast<void**>(&ps->d_table[dt]), bytes);
        if (e == hipSuccess) e = hipMemcpy(ps->d_table[dt], tab.data(), bytes, hipMemcpyHostToDevice);
        if (e != hipSuccess) break;
        std::vector<uint32_t> owner(ps->total_tiles[dt]);
        for (size_t i = 0; i < tab.size(); ++i) {
            const uint64_t end = i + 1 < tab.size() ? tab[i + 1].tile_begin : ps->total_tiles[dt];
            for (uint64_t tl = tab[i].tile_begin; tl < end; ++tl) owner[tl] = static_cast<uint32_t>(i);
        }
        e = hipMalloc(reinterpret_cast<void**>(&ps->d_tile_tensor[dt]), owner.size() * sizeof(uint32_t));
        if (e == hipSuccess)
            e = hipMemcpy(ps->d_tile_tensor[dt], owner.data(), owner.size() * sizeof(uint32_t),
                          hipMemcpyHostToDevice);
    }
    for (size_t i = 0; i < mezo_paramset::kUses && e == hipSuccess; ++i)
        e = hipEventCreateWithFlags(&ps->uses[i].done, hipEventDisableTiming);
    if (e == hipSuccess) {
        const std::vector<unsigned long long> zeros(2 * mezo_paramset::kCkPairs, 0ull);
        e = hipMalloc(reinterpret_cast<void**>(&ps->d_ck), zeros.size() * sizeof(zeros[0]));
        if (e == hipSuccess)
            e = hipMemcpy(ps->d_ck, zeros.data(), zeros.size() * sizeof(zeros[0]), hipMemcpyHostToDevice);
    }
    // the device address of mezo_replay_noalloc's staging array, resolved at
    // set-up (once per device, cached), so that entry point makes no such
    // query itself, also not under graph capture
    mezo::SeedRec* staging = nullptr;
    if (e == hipSuccess) e = mezo::noalloc_scratch(&staging);
    if (e != hipSuccess) {
        for (int dt = 0; dt < mezo_paramset::kTypes; ++dt) {
            if (ps->d_table[dt]) (void)hipFree(ps->d_table[dt]);
            if (ps->d_tile_tensor[dt]) (void)hipFree(ps->d_tile_tensor[dt]);
            ps->d_table[dt] = nullptr;
            ps->d_tile_tensor[dt] = nullptr;
        }
        for (auto& u : ps->uses) {
            if (u.done) (void)hipEventDestroy(u.done);
            u.done = nullptr;
        }
        if (ps->d_ck) (void)hipFree(ps->d_ck);
        ps->d_ck = nullptr;
        return hip_fail(e, "paramset device table");
    }
    ps->device = dev;
    return MEZO_OK;
}

// Whether work enqueued on stream is being captured into a graph (then it
// runs only when the graph is launched, possibly many times).
int capturing(hipStream_t stream, bool& out)
{
    hipStreamCaptureStatus st = hipStreamCaptureStatusNone;
    MEZO_HIP(hipStreamIsCapturing(stream, &st));
    out = st != hipStreamCaptureStatusNone;
    return MEZO_OK;
}

// A paramset's first call creates its device tables (allocations and
// copies), which a graph capture cannot record.
int refuse_first_use_in_capture(const mezo_paramset* ps)
{
    if (ps->device >= 0) return MEZO_OK;
    set_error("a paramset's first call allocates its device tables and cannot be captured into a graph");
    return MEZO_EINVAL;
}

// The use entry of stream: its own, else one not used yet (seq 0), else the
// one used longest ago, taken over after its work has completed (a host wait).
int use_entry(mezo_paramset* ps, hipStream_t stream, mezo_paramset::Use*& out)
{
    mezo_paramset::Use* use = nullptr;
    for (auto& u : ps->uses)
        if (u.seq && u.stream == stream) use = &u;
    if (!use) {
        use = std::min_element(std::begin(ps->uses), std::end(ps->uses),
                               [](const mezo_paramset::Use& a, const mezo_paramset::Use& b) { return a.seq < b.seq; });
        if (use->seq) MEZO_HIP(hipEventSynchronize(use->done));
        use->stream = stream;
    }
    out = use;
    return MEZO_OK;
}

// Record that ps's tables are read by work enqueued so far on stream, in its
// use entry (after ensure_device: the events exist; nothing is created here).
int record_use(mezo_paramset* ps, mezo_paramset::Use* use, hipStream_t stream)
{
    use->seq = ++ps->use_seq;
    MEZO_HIP(hipEventRecord(use->done, stream));
    return MEZO_OK;
}

int mark_use(mezo_paramset* ps, hipStream_t stream)
{
    mezo_paramset::Use* use = nullptr;
    const int rc = use_entry(ps, stream, use);
    return rc ? rc : record_use(ps, use, stream);
}

// Records one engine launch applies at most when a call can split its list
// at step ends (a replay): a long catch-up then runs as launches of bounded
// length instead of one kernel of arbitrary length.
constexpr size_t kMaxLaunchRecords = size_t(1) << 16;

// A run of records of a call: [data, data + size).
struct RecSpan {
    const mezo::SeedRec* data;
    size_t size;
    bool empty() const { return size == 0; }
};

// One engine launch per storage type of ps with the records args carries
// (src: read that set, of the same layout, and write ps).
hipError_t launch_tables(const mezo_paramset* ps, mezo::EngineArgs& args, bool portable, hipStream_t stream,
                         const mezo_paramset* src)
{
    hipError_t e = hipSuccess;
    for (uint32_t dt = 0; dt < mezo::kStorageTypes && e == hipSuccess; ++dt) {
        if (ps->table[dt].empty()) continue;
        args.tensors = ps->d_table[dt];
        args.tile_tensor = ps->d_tile_tensor[dt];
        args.src_tensors = src ? src->d_table[dt] : nullptr;
        args.n_tensors = static_cast<uint32_t>(ps->table[dt].size());
        args.total_tiles = ps->total_tiles[dt];
        e = dt == mezo::kNF4 ? mezo::launch_engine_nf4(args, portable, stream)
                             : mezo::launch_engine_dense(args, dt, portable, stream);
    }
    return e;
}

// Enqueue the engine over every storage type of ps, with the Gaussian the
// records were made for. With src (same layout), read src and write ps; that
// launch is made even with no records (a copy).
int launch_records(mezo_paramset* ps, RecSpan recs, bool portable, hipStream_t stream,
                   mezo_paramset* src = nullptr)
{
    if (recs.empty() && !src) return MEZO_OK;
    if (recs.size > UINT32_MAX) return MEZO_ERANGE;  // the kernels count records in 32 bits
    bool capture = false;
    int rc = capturing(stream, capture);
    if (rc) return rc;
    if (capture) {
        rc = refuse_first_use_in_capture(ps);
        if (rc == MEZO_OK && src) rc = refuse_first_use_in_capture(src);
        if (rc) return rc;
        if (recs.size > mezo::kInlineRecs) {
            // a graph would copy the records from a host slot that later
            // calls reuse
            set_error("record lists longer than 32 are staged through host memory and cannot be captured");
            return MEZO_EINVAL;
        }
    }
    rc = ensure_device(ps);
    if (rc) return rc;
    if (src && src != ps) {
        rc = ensure_device(src);
        if (rc) return rc;
        if (src->device != ps->device) {
            set_error("source and destination paramsets live on different devices");
            return MEZO_EINVAL;
        }
    }
    mezo::EngineArgs args;
    std::memset(&args, 0, sizeof(args));
    args.n_rec = static_cast<uint32_t>(recs.size);
    mezo_paramset::Slot* slot = nullptr;
    if (recs.size <= mezo::kInlineRecs) {
        std::copy(recs.data, recs.data + recs.size, args.inl);
    } else {
        slot = &ps->slots[ps->next_slot++ % mezo_paramset::kSlots];
        if (slot->done)
            MEZO_HIP(hipEventSynchronize(slot->done));
        else
            MEZO_HIP(hipEventCreateWithFlags(&slot->done, hipEventDisableTiming));
        if (slot->cap < recs.size) {
            size_t cap = std::max<size_t>(recs.size, 2 * slot->cap);
            if (slot->host) MEZO_HIP(hipHostFree(slot->host));
            if (slot->dev) MEZO_HIP(hipFree(slot->dev));
            slot->host = nullptr;
            slot->dev = nullptr;
            slot->cap = 0;
            MEZO_HIP(hipHostMalloc(reinterpret_cast<void**>(&slot->host), cap * sizeof(mezo::SeedRec)));
            MEZO_HIP(hipMalloc(reinterpret_cast<void**>(&slot->dev), cap * sizeof(mezo::SeedRec)));
            slot->cap = cap;
        }
        std::memcpy(slot->host, recs.data, recs.size * sizeof(mezo::SeedRec));
        MEZO_HIP(hipMemcpyAsync(slot->dev, slot->host, recs.size * sizeof(mezo::SeedRec),
                                hipMemcpyHostToDevice, stream));
        args.ext = slot->dev;
    }
    hipError_t e = launch_tables(ps, args, portable, stream, src);
    // The slot is reused only after this event: recorded whenever its copy
    // was enqueued, also when a launch failed.
    if (slot) {
        const hipError_t er = hipEventRecord(slot->done, stream);
        if (e == hipSuccess) e = er;
    }
    if (e != hipSuccess) return hip_fail(e, "engine launch");
    if (capture) return MEZO_OK;  // a graph's launches are the caller's to wait for
    rc = mark_use(ps, stream);
    if (rc == MEZO_OK && src && src != ps) rc = mark_use(src, stream);
    return rc;
}

int launch_records(mezo_paramset* ps, const std::vector<mezo::SeedRec>& recs, bool portable, hipStream_t stream,
                   mezo_paramset* src = nullptr)
{
    return launch_records(ps, RecSpan{recs.data(), recs.size()}, portable, stream, src);
}

// Byte ranges [begin, end) of device memory a tensor occupies.
using Span = std::pair<uint64_t, uint64_t>;

uint64_t nf4_code_bytes(uint64_t n) { return (n + 1) / 2; }
uint64_t nf4_absmax_bytes(uint64_t n) { return 4 * ((n + MEZO_NF4_BLOCK - 1) / MEZO_NF4_BLOCK); }

void add_spans(uint64_t data, uint64_t aux, uint64_t numel, uint32_t dtype, std::vector<Span>& out)
{
    if (dtype == MEZO_NF4) {
        out.emplace_back(data, data + nf4_code_bytes(numel));
        out.emplace_back(aux, aux + nf4_absmax_bytes(numel));
    } else {
        out.emplace_back(data, data + numel * (dtype == MEZO_F32 ? 4 : 2));
    }
}

bool disjoint(std::vector<Span>& spans)
{
    std::sort(spans.begin(), spans.end());
    uint64_t reach = 0;
    for (const auto& sp : spans) {
        if (sp.first < reach) return false;
        reach = std::max(reach, sp.second);
    }
    return true;
}

uint64_t tile_of(uint32_t dtype)
{
    return dtype == MEZO_F32 ? mezo::kTileF32 : (dtype == MEZO_BF16 ? mezo::kTileBF16 : mezo::kTileNF4);
}

// dst and src describe the same tensors (count, ids, sizes, offsets, storage types, in
// registration order per storage type) and share no memory except where a
// tensor is its own source.
int check_pair(const mezo_paramset* dst, const mezo_paramset* src)
{
    if (dst == src) return MEZO_OK;
    std::vector<Span> spans;
    for (int dt = 0; dt < mezo_paramset::kTypes; ++dt) {
        const auto& a = dst->table[dt];
        const auto& b = src->table[dt];
        if (a.size() != b.size()) return MEZO_EINVAL;
        for (size_t i = 0; i < a.size(); ++i) {
            if (a[i].numel != b[i].numel || a[i].tensor_id != b[i].tensor_id || a[i].first != b[i].first)
                return MEZO_EINVAL;
            const bool same = b[i].data == a[i].data && b[i].aux == a[i].aux;
            add_spans(a[i].data, a[i].aux, a[i].numel, a[i].dtype, spans);
            if (!same) add_spans(b[i].data, b[i].aux, b[i].numel, b[i].dtype, spans);
        }
    }
    return disjoint(spans) ? MEZO_OK : MEZO_EOVERLAP;
}

}  // namespace

extern "C" {

int mezo_paramset_create(const mezo_tensor_t* t, uint32_t n, mezo_paramset_t* out)
{
    return guarded("mezo_paramset_create", [&]() -> int {
        if (!t || !out || n == 0) return MEZO_EINVAL;
        std::vector<Span> spans;
        std::vector<uint32_t> ids;
        spans.reserve(2 * size_t(n));
        ids.reserve(n);
        for (uint32_t i = 0; i < n; ++i) {
            if (t[i].dtype != MEZO_F32 && t[i].dtype != MEZO_BF16 && t[i].dtype != MEZO_NF4) return MEZO_EDTYPE;
            if (!t[i].data || (reinterpret_cast<uintptr_t>(t[i].data) & 15u)) return MEZO_EINVAL;
            if (t[i].numel == 0 || t[i].numel > MEZO_MAX_NUMEL) return MEZO_EINVAL;
            // a shard's first element: block-aligned, inside the counter's range
            if ((t[i].first & 7u) || t[i].first > MEZO_MAX_NUMEL - t[i].numel) return MEZO_EINVAL;
            if (t[i].dtype == MEZO_NF4 && t[i].first != 0) return MEZO_EINVAL;
            if (t[i].dtype == MEZO_NF4) {
                if (!t[i].absmax || (reinterpret_cast<uintptr_t>(t[i].absmax) & 15u)) return MEZO_EINVAL;
            } else if (t[i].absmax) {
                return MEZO_EINVAL;
            }
            add_spans(reinterpret_cast<uint64_t>(t[i].data), reinterpret_cast<uint64_t>(t[i].absmax), t[i].numel,
                      t[i].dtype, spans);
            ids.push_back(t[i].tensor_id);
        }
        std::sort(ids.begin(), ids.end());
        if (std::adjacent_find(ids.begin(), ids.end()) != ids.end()) return MEZO_EINVAL;
        if (!disjoint(spans)) return MEZO_EOVERLAP;

        std::unique_ptr<mezo_paramset> ps(new mezo_paramset);
        uint64_t numel = 0;
        for (uint32_t i = 0; i < n; ++i) {
            const uint32_t dt = t[i].dtype;
            mezo::TensorDesc d;
            d.data = reinterpret_cast<uint64_t>(t[i].data);
            d.aux = reinterpret_cast<uint64_t>(t[i].absmax);
            d.numel = t[i].numel;
            d.tensor_id = t[i].tensor_id;
            d.dtype = dt;
            d.first = t[i].first;
            d.tile_begin = ps->total_tiles[dt];
            const uint64_t per = tile_of(dt);
            ps->total_tiles[dt] += (t[i].numel + per - 1) / per;
            ps->table[dt].push_back(d);
            numel += t[i].numel;
        }
        ps->numel = numel;
        for (int dt = 0; dt < mezo_paramset::kTypes; ++dt) {
            if (ps->total_tiles[dt] > 0x7FFFFFFFull) return MEZO_EINVAL;  // more tiles than one launch can address
        }
        *out = ps.release();
        return MEZO_OK;
    });
}

void mezo_paramset_destroy(mezo_paramset_t ps)
{
    if (!ps) return;
    {
        // taken so that a call still running on another thread finishes
        // first; the caller must not start new ones
        std::unique_lock<std::mutex> lock(ps->mu, std::defer_lock);
        try {
            lock.lock();
        } catch (...) {
        }
        for (auto& u : ps->uses) {
            if (!u.done) continue;
            if (u.seq) (void)hipEventSynchronize(u.done);
            (void)hipEventDestroy(u.done);
        }
        for (auto& s : ps->slots) {
            if (s.done) {
                (void)hipEventSynchronize(s.done);
                (void)hipEventDestroy(s.done);
            }
            if (s.host) (void)hipHostFree(s.host);
            if (s.dev) (void)hipFree(s.dev);
        }
        for (int dt = 0; dt < mezo_paramset::kTypes; ++dt) {
            if (ps->d_table[dt]) (void)hipFree(ps->d_table[dt]);
            if (ps->d_tile_tensor[dt]) (void)hipFree(ps->d_tile_tensor[dt]);
        }
        if (ps->d_ck) (void)hipFree(ps->d_ck);
    }
    delete ps;
}

uint64_t mezo_paramset_numel(mezo_paramset_t ps) { return ps ? ps->numel : 0; }

int mezo_paramset_set_gaussian(mezo_paramset_t ps, uint32_t gaussian)
{
    if (!ps || (gaussian != MEZO_GAUSS_FAST && gaussian != MEZO_GAUSS_PORTABLE)) return MEZO_EINVAL;
    ps->gaussian.store(gaussian);
    return MEZO_OK;
}

int mezo_perturb(mezo_paramset_t ps, mezo_seed_t seed, float scale, void* stream)
{
    return guarded("mezo_perturb", [&]() -> int {
        if (!ps) return MEZO_EINVAL;
        if (!std::isfinite(scale)) return MEZO_ERANGE;
        if (scale == 0.0f) return MEZO_OK;
        const bool portable = portable_of(ps);
        std::vector<mezo::SeedRec> recs(1, make_rec(seed, scale, true, !portable));
        std::lock_guard<std::mutex> lock(ps->mu);
        return launch_records(ps, recs, portable, static_cast<hipStream_t>(stream));
    });
}

int mezo_perturb_multi(mezo_paramset_t ps, const mezo_seed_t* seeds, const float* scales, uint32_t n,
                       void* stream)
{
    return guarded("mezo_perturb_multi", [&]() -> int {
        if (!ps) return MEZO_EINVAL;
        if (n == 0) return MEZO_OK;
        if (!seeds || !scales) return MEZO_EINVAL;
        for (uint32_t i = 0; i < n; ++i)
            if (!std::isfinite(scales[i])) return MEZO_ERANGE;
        const bool portable = portable_of(ps);
        std::vector<mezo::SeedRec> recs;
        recs.reserve(n);
        for (uint32_t i = 0; i < n; ++i)
            if (scales[i] != 0.0f) recs.push_back(make_rec(seeds[i], scales[i], true, !portable));
        std::lock_guard<std::mutex> lock(ps->mu);
        return launch_records(ps, recs, portable, static_cast<hipStream_t>(stream));
    });
}

int mezo_update_multi(mezo_paramset_t ps, const mezo_seed_t* seeds, const int8_t* q, uint32_t K,
                      const mezo_codec_t* codec, float lr, void* stream)
{
    return guarded("mezo_update_multi", [&]() -> int {
        if (!ps) return MEZO_EINVAL;
        const bool portable = portable_of(ps);
        std::vector<mezo::SeedRec> recs;
        recs.reserve(K);
        int rc = append_step(seeds, q, K, codec, lr, !portable, recs);
        if (rc) return rc;
        std::lock_guard<std::mutex> lock(ps->mu);
        return launch_records(ps, recs, portable, static_cast<hipStream_t>(stream));
    });
}

int mezo_perturb_from(mezo_paramset_t dst, mezo_paramset_t src, mezo_seed_t seed, float scale,
                      void* stream)
{
    return guarded("mezo_perturb_from", [&]() -> int {
        if (!dst || !src) return MEZO_EINVAL;
        if (!std::isfinite(scale)) return MEZO_ERANGE;
        int rc = check_pair(dst, src);
        if (rc) return rc;
        const bool portable = portable_of(dst);
        std::vector<mezo::SeedRec> recs;
        if (scale != 0.0f) recs.push_back(make_rec(seed, scale, true, !portable));
        if (dst == src) {
            std::lock_guard<std::mutex> lock(dst->mu);
            return launch_records(dst, recs, portable, static_cast<hipStream_t>(stream));
        }
        std::scoped_lock lock(dst->mu, src->mu);
        return launch_records(dst, recs, portable, static_cast<hipStream_t>(stream), src);
    });
}

int mezo_update_multi_from(mezo_paramset_t dst, mezo_paramset_t src, const mezo_seed_t* seeds,
                           const int8_t* q, uint32_t K, const mezo_codec_t* codec, float lr, void* stream)
{
    return guarded("mezo_update_multi_from", [&]() -> int {
        if (!dst || !src) return MEZO_EINVAL;
        const bool portable = portable_of(dst);
        std::vector<mezo::SeedRec> recs;
        recs.reserve(K);
        int rc = append_step(seeds, q, K, codec, lr, !portable, recs);
        if (rc) return rc;
        rc = check_pair(dst, src);
        if (rc) return rc;
        if (dst == src) {
            std::lock_guard<std::mutex> lock(dst->mu);
            return launch_records(dst, recs, portable, static_cast<hipStream_t>(stream));
        }
        std::scoped_lock lock(dst->mu, src->mu);
        return launch_records(dst, recs, portable, static_cast<hipStream_t>(stream), src);
    });
}

int mezo_replay(mezo_paramset_t ps, const mezo_step_t* steps, uint32_t T, const mezo_codec_t* codec,
                void* stream)
{
    return guarded("mezo_replay", [&]() -> int {
        if (!ps || !codec) return MEZO_EINVAL;
        if (!codec_valid(codec)) return MEZO_ERANGE;
        if (T == 0) return MEZO_OK;
        if (!steps) return MEZO_EINVAL;
        const bool portable = portable_of(ps);
        std::vector<mezo::SeedRec> recs;
        uint64_t total = 0;
        for (uint32_t t = 0; t < T; ++t) total += steps[t].K;
        if (total > UINT32_MAX) return MEZO_ERANGE;  // the kernels count records in 32 bits
        recs.reserve(total);
        std::vector<size_t> step_ends;  // record count after each step that kept records
        for (uint32_t t = 0; t < T; ++t) {
            const size_t before = recs.size();
            int rc = append_step(steps[t].seeds, steps[t].q, steps[t].K, codec, steps[t].lr, !portable, recs);
            if (rc) return rc;
            if (recs.size() > before) step_ends.push_back(recs.size());
        }
        // launches of at most kMaxLaunchRecords records, split at step ends
        // (where every step rounds to storage anyway: the result is the same);
        // a longer single step runs alone
        std::lock_guard<std::mutex> lock(ps->mu);
        const hipStream_t st = static_cast<hipStream_t>(stream);
        size_t start = 0, end = 0;
        for (size_t e : step_ends) {
            if (e - start > kMaxLaunchRecords && end > start) {
                int rc = launch_records(ps, RecSpan{recs.data() + start, end - start}, portable, st);
                if (rc) return rc;
                start = end;
            }
            end = e;
        }
        return launch_records(ps, RecSpan{recs.data() + start, end - start}, portable, st);
    });
}

int mezo_replay_noalloc(mezo_paramset_t ps, const mezo_step_t* steps, uint32_t T, const mezo_codec_t* codec,
                        void* stream)
{
    // Nothing below allocates: records are built in a fixed array on the
    // stack and reach the device through the file-scope staging array
    // (noalloc.hip), or the kernel arguments for at most 32 records.
    return guarded("mezo_replay_noalloc", [&]() -> int {
        if (!ps || !codec) return MEZO_EINVAL;
        if (!codec_valid(codec)) return MEZO_ERANGE;
        if (T == 0) return MEZO_OK;
        if (!steps) return MEZO_EINVAL;
        uint64_t total = 0;  // records kept (non-zero weights)
        for (uint32_t t = 0; t < T; ++t) {
            const int rc = check_step(steps[t].seeds, steps[t].q, steps[t].K, codec, steps[t].lr);
            if (rc) return rc;
            for (uint32_t k = 0; k < steps[t].K; ++k) total += step_coef(steps[t].q[k], *codec, steps[t].lr) != 0.0f;
        }
        if (total == 0) return MEZO_OK;
        if (total > mezo::kNoAllocRecords) {
            set_error("mezo_replay_noalloc", "more than 65536 records (non-zero terms) in one call");
            return MEZO_ERANGE;
        }
        const bool portable = portable_of(ps);
        const hipStream_t st = static_cast<hipStream_t>(stream);
        std::lock_guard<std::mutex> lock(ps->mu);
        int dev = -1;
        MEZO_HIP(hipGetDevice(&dev));
        if (ps->device < 0) {
            set_error("mezo_replay_noalloc",
                      "the paramset has no device tables yet: its first call must be one that may allocate them");
            return MEZO_EINVAL;
        }
        if (ps->device != dev) {
            set_error("paramset used on a device other than the one it was first used on");
            return MEZO_EINVAL;
        }
        bool capture = false;
        int rc = capturing(st, capture);
        if (rc) return rc;
        mezo::EngineArgs args;
        std::memset(&args, 0, sizeof(args));
        args.n_rec = static_cast<uint32_t>(total);
        if (total <= mezo::kInlineRecs) {
            uint32_t i = 0;
            for (uint32_t t = 0; t < T; ++t)
                if (steps[t].K)
                    emit_step(steps[t].seeds, steps[t].q, steps[t].K, *codec, steps[t].lr, !portable,
                              [&](const mezo::SeedRec& r) { args.inl[i++] = r; });
        } else {
            mezo::SeedRec* scratch = nullptr;
            MEZO_HIP(mezo::noalloc_scratch(&scratch));
            mezo::SeedRec chunk[mezo::kStageRecs];
            uint32_t n = 0, offset = 0;
            hipError_t e = hipSuccess;
            const auto flush = [&]() {
                if (n && e == hipSuccess) e = mezo::launch_stage(scratch, offset, chunk, n, st);
                offset += n;
                n = 0;
            };
            for (uint32_t t = 0; t < T; ++t)
                if (steps[t].K)
                    emit_step(steps[t].seeds, steps[t].q, steps[t].K, *codec, steps[t].lr, !portable,
                              [&](const mezo::SeedRec& r) {
                                  chunk[n++] = r;
                                  if (n == mezo::kStageRecs) flush();
                              });
            flush();
            if (e != hipSuccess) return hip_fail(e, "record staging");
            args.ext = scratch;
        }
        const hipError_t e = launch_tables(ps, args, portable, st, nullptr);
        if (e != hipSuccess) return hip_fail(e, "engine launch");
        return capture ? MEZO_OK : mark_use(ps, st);
    });
}

int mezo_checksum(mezo_paramset_t ps, uint64_t* out_dev, void* stream)
{
    return guarded("mezo_checksum", [&]() -> int {
        if (!ps || !out_dev || (reinterpret_cast<uintptr_t>(out_dev) & 7u)) return MEZO_EINVAL;
        std::lock_guard<std::mutex> lock(ps->mu);
        hipStream_t st = static_cast<hipStream_t>(stream);
        bool capture = false;
        int rc = capturing(st, capture);
        if (rc == MEZO_OK && capture) rc = refuse_first_use_in_capture(ps);
        if (rc) return rc;
        rc = ensure_device(ps);
        if (rc) return rc;
        mezo::ChecksumArgs tabs[mezo_paramset::kTypes] = {};
        uint32_t dts[mezo_paramset::kTypes];
        int n = 0;
        for (uint32_t dt = 0; dt < mezo::kStorageTypes; ++dt) {
            if (ps->table[dt].empty()) continue;
            tabs[n].tensors = ps->d_table[dt];
            tabs[n].tile_tensor = ps->d_tile_tensor[dt];
            tabs[n].total_tiles = ps->total_tiles[dt];
            dts[n] = dt;
            ++n;
        }
        // the running sum of the stream's use entry (captured: the graphs' own)
        mezo_paramset::Use* use = nullptr;
        size_t pair = mezo_paramset::kUses;
        if (!capture) {
            rc = use_entry(ps, st, use);
            if (rc) return rc;
            pair = static_cast<size_t>(use - ps->uses);
        }
        MEZO_HIP(mezo::launch_checksum(tabs, dts, n, reinterpret_cast<unsigned long long*>(out_dev),
                                       ps->d_ck + 2 * pair, ps->device, st));
        return capture ? MEZO_OK : record_use(ps, use, st);
    });
}

namespace {
int nf4_convert(const void* values, uint32_t dtype, uint64_t n, const void* codes, const float* absmax,
                bool quantize, void* stream)
{
    if (dtype != MEZO_F32 && dtype != MEZO_BF16) return MEZO_EDTYPE;
    if (!values || !codes || !absmax || n == 0 || n > MEZO_MAX_NUMEL) return MEZO_EINVAL;
    const uint64_t v = reinterpret_cast<uint64_t>(values);
    const uint64_t c = reinterpret_cast<uint64_t>(codes);
    const uint64_t a = reinterpret_cast<uint64_t>(absmax);
    if ((v | c | a) & 15u) return MEZO_EINVAL;
    std::vector<Span> spans;
    add_spans(v, 0, n, dtype, spans);
    add_spans(c, a, n, MEZO_NF4, spans);
    if (!disjoint(spans)) return MEZO_EOVERLAP;
    mezo::NF4ConvArgs args;
    args.values = v;
    args.codes = c;
    args.absmax = a;
    args.n = n;
    args.dtype = dtype;
    MEZO_HIP(mezo::launch_nf4(args, quantize, static_cast<hipStream_t>(stream)));
    return MEZO_OK;
}
}  // namespace

int mezo_nf4_quantize(const void* src, uint32_t src_dtype, uint64_t n, void* codes, float* absmax, void* stream)
{
    return guarded("mezo_nf4_quantize", [&] { return nf4_convert(src, src_dtype, n, codes, absmax, true, stream); });
}

int mezo_nf4_dequantize(const void* codes, const float* absmax, uint64_t n, void* dst, uint32_t dst_dtype,
                        void* stream)
{
    return guarded("mezo_nf4_dequantize",
                   [&] { return nf4_convert(dst, dst_dtype, n, codes, absmax, false, stream); });
}

int quantize_projgrad(const float* g, int8_t* q, uint32_t n, const mezo_codec_t* codec)
{
    if (!codec) return MEZO_EINVAL;
    if (!codec_valid(codec)) return MEZO_ERANGE;
    if (n == 0) return MEZO_OK;
    if (!g || !q) return MEZO_EINVAL;
    for (uint32_t i = 0; i < n; ++i)
        if (std::isnan(g[i])) return MEZO_ERANGE;
    const double qmax = code_max(*codec);
    for (uint32_t i = 0; i < n; ++i) q[i] = encode(g[i], *codec, qmax);
    return MEZO_OK;
}

int mezo_dequantize(const int8_t* q, float* g, uint32_t n, const mezo_codec_t* codec)
{
    if (!codec) return MEZO_EINVAL;
    if (!codec_valid(codec)) return MEZO_ERANGE;
    if (n == 0) return MEZO_OK;
    if (!g || !q) return MEZO_EINVAL;
    const int qmax = code_max(*codec);
    for (uint32_t i = 0; i < n; ++i)
        if (q[i] > qmax || q[i] < -qmax) return MEZO_ERANGE;  // -128 included
    for (uint32_t i = 0; i < n; ++i) g[i] = decode(q[i], *codec);
    return MEZO_OK;
}

int mezo_debug_generate(mezo_seed_t seed, uint32_t tensor_id, uint64_t first_elem, uint64_t count,
                        uint32_t gaussian, uint32_t* words_dev, float* z_dev, void* stream)
{
    if (first_elem > MEZO_MAX_NUMEL || count > MEZO_MAX_NUMEL - first_elem) return MEZO_EINVAL;
    if (gaussian != MEZO_GAUSS_FAST && gaussian != MEZO_GAUSS_PORTABLE) return MEZO_EINVAL;
    if (count == 0 || (!words_dev && !z_dev)) return MEZO_OK;
    mezo::GenArgs a;
    std::memset(&a, 0, sizeof(a));
    a.rec = make_rec(seed, 0.0f, false, false);
    a.portable = gaussian == MEZO_GAUSS_PORTABLE ? 1u : 0u;
    a.tensor_id = tensor_id;
    a.first = first_elem;
    a.count = count;
    a.words = words_dev;
    a.z = z_dev;
    MEZO_HIP(mezo::launch_generate(a, static_cast<hipStream_t>(stream)));
    return MEZO_OK;
}

int mezo_debug_box_muller(const uint32_t* words_dev, uint64_t n_blocks, uint32_t gaussian, float* z_dev,
                          void* stream)
{
    if (gaussian != MEZO_GAUSS_FAST && gaussian != MEZO_GAUSS_PORTABLE) return MEZO_EINVAL;
    if (n_blocks == 0) return MEZO_OK;
    if (!words_dev || !z_dev || n_blocks > (uint64_t(1) << 32)) return MEZO_EINVAL;
    if ((reinterpret_cast<uintptr_t>(words_dev) | reinterpret_cast<uintptr_t>(z_dev)) & 15u) return MEZO_EINVAL;
    MEZO_HIP(mezo::launch_box_muller(words_dev, n_blocks, gaussian == MEZO_GAUSS_PORTABLE ? 1u : 0u, z_dev,
                                     static_cast<hipStream_t>(stream)));
    return MEZO_OK;
}

const char* mezo_strerror(int code)
{
    switch (code) {
    case MEZO_OK: return "success";
    case MEZO_EINVAL: return "invalid argument (null/misaligned pointer, bad size or duplicate tensor id)";
    case MEZO_EDTYPE: return "unknown storage type";
    case MEZO_EOVERLAP: return "tensors overlap in memory";
    case MEZO_EORDER: return "seeds not strictly ascending by (machine, step, sample)";
    case MEZO_ERANGE: return "value out of range (q = -128, NaN gradient, non-finite lr/scale, bad codec)";
    case MEZO_EHIP: return "HIP runtime failure";
    case MEZO_ENOMEM: return "host memory allocation failed";
    default: return "unknown error code";
    }
}

const char* mezo_last_error(void) { return t_last_error; }

int mezo_version(void) { return 500; }

}  // extern "C"
