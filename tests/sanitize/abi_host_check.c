/* abi_host_check.c — TEST INFRASTRUCTURE ONLY: drives the host code of the C
 * ABI (api.cpp, built with AddressSanitizer and UndefinedBehaviorSanitizer)
 * through the HIP stand-in of hip_double.cpp, on a machine without a GPU.
 *
 * Covers what the host code decides on its own: argument checks and their
 * error codes, overlap and layout checks, seed ordering, the one-byte codec
 * (Section 3) over every code, the records a call hands to the engine
 * (coefficients, zero terms dropped, step ends flagged), staging of long
 * record lists through the slot ring and its growth, replay split at step
 * ends, per-stream event bookkeeping, device and graph-capture refusals, a
 * failed device allocation, and concurrent callers. Every paramset is
 * destroyed at the end, and every "device" allocation and event must be gone.
 * Exit status 0 when every check passed. */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "mezo.h"

/* control and inspection of the HIP stand-in */
void double_set_device(int d);
void double_set_capturing(int on);
void double_fail_malloc_in(long n);
unsigned long double_engine_launches(uint32_t dtype);
unsigned long double_checksum_launches(void);
unsigned long double_nf4_launches(void);
unsigned long double_generate_launches(void);
unsigned long double_event_syncs(void);
unsigned long double_events_live(void);
size_t double_device_allocations(void);
unsigned long double_allocation_calls(void);
unsigned long double_stage_launches(void);
uint32_t double_last_records(float* coef, uint32_t* last, uint32_t* machine, uint32_t max);
int double_last_out_of_place(void);

static int g_checks, g_failed;

#define CHECK(cond)                                                                 \
    do {                                                                            \
        ++g_checks;                                                                 \
        if (!(cond)) {                                                              \
            ++g_failed;                                                             \
            fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond); \
        }                                                                           \
    } while (0)

#define MAXREC 80000
static float g_coef[MAXREC];
static uint32_t g_last[MAXREC], g_mach[MAXREC];

static mezo_tensor_t T(uintptr_t data, uint64_t n, uint32_t id, uint32_t dt, uintptr_t absmax, uint64_t first)
{
    mezo_tensor_t t;
    t.data = (void*)data;
    t.numel = n;
    t.tensor_id = id;
    t.dtype = dt;
    t.absmax = (void*)absmax;
    t.first = first;
    return t;
}

static int create1(mezo_tensor_t t, mezo_paramset_t* ps) { return mezo_paramset_create(&t, 1, ps); }

static mezo_seed_t S(uint64_t m, uint32_t step, uint32_t sample)
{
    mezo_seed_t s;
    s.machine = m;
    s.step = step;
    s.sample = sample;
    return s;
}

static void check_create(void)
{
    mezo_paramset_t ps = NULL;
    mezo_tensor_t two[3];
    CHECK(mezo_paramset_create(NULL, 1, &ps) == MEZO_EINVAL);
    CHECK(create1(T(0, 16, 0, MEZO_F32, 0, 0), &ps) == MEZO_EINVAL);
    CHECK(create1(T(0x1004, 16, 0, MEZO_F32, 0, 0), &ps) == MEZO_EINVAL);
    CHECK(create1(T(0x1000, 0, 0, MEZO_F32, 0, 0), &ps) == MEZO_EINVAL);
    CHECK(create1(T(0x1000, MEZO_MAX_NUMEL + 1, 0, MEZO_F32, 0, 0), &ps) == MEZO_EINVAL);
    CHECK(create1(T(0x1000, 16, 0, 5, 0, 0), &ps) == MEZO_EDTYPE);
    CHECK(create1(T(0x1000, 16, 0, MEZO_NF4, 0, 0), &ps) == MEZO_EINVAL);
    CHECK(create1(T(0x1000, 16, 0, MEZO_NF4, 0x2008, 0), &ps) == MEZO_EINVAL);
    CHECK(create1(T(0x1000, 16, 0, MEZO_F32, 0x2000, 0), &ps) == MEZO_EINVAL);
    CHECK(create1(T(0x1000, 16, 0, MEZO_NF4, 0x1000, 0), &ps) == MEZO_EOVERLAP);
    CHECK(create1(T(0x1000, 16, 0, MEZO_F32, 0, 4), &ps) == MEZO_EINVAL);
    CHECK(create1(T(0x1000, 16, 0, MEZO_F32, 0, MEZO_MAX_NUMEL - 8), &ps) == MEZO_EINVAL);
    CHECK(create1(T(0x1000, 16, 0, MEZO_NF4, 0x2000, 64), &ps) == MEZO_EINVAL);
    two[0] = T(0x1000, 16, 3, MEZO_F32, 0, 0);
    two[1] = T(0x2000, 16, 3, MEZO_F32, 0, 0);
    CHECK(mezo_paramset_create(two, 2, &ps) == MEZO_EINVAL);
    two[1] = T(0x1030, 16, 1, MEZO_F32, 0, 0);
    CHECK(mezo_paramset_create(two, 2, &ps) == MEZO_EOVERLAP);
    two[0] = T(0x1000, 260, 0, MEZO_NF4, 0x2000, 0);  /* 5 absmax values = 20 B */
    two[1] = T(0x2010, 4, 1, MEZO_F32, 0, 0);
    CHECK(mezo_paramset_create(two, 2, &ps) == MEZO_EOVERLAP);
    CHECK(ps == NULL);
    two[0] = T(0x1000, 32, 0, MEZO_NF4, 0x3000, 0);
    two[1] = T(0x1010, 4, 1, MEZO_F32, 0, 0);
    two[2] = T(0x3010, 8, 2, MEZO_BF16, 0, 0);
    CHECK(mezo_paramset_create(two, 3, &ps) == MEZO_OK);
    CHECK(mezo_paramset_numel(ps) == 44);
    mezo_paramset_destroy(ps);
    mezo_paramset_destroy(NULL);
}

static void check_codec(void)
{
    const float alphas[3] = {1.4426950408889634f, 1.0f, 3.0f};
    mezo_codec_t c;
    int8_t q[255], q2[255];
    float g[255];
    int i, a;
    c.kind = MEZO_CODEC_LINEAR;
    c.scale = 1.0f / 127.0f;
    c.alpha = 0.0f;
    for (i = 0; i < 255; ++i) q[i] = (int8_t)(i - 127);
    CHECK(mezo_dequantize(q, g, 255, &c) == MEZO_OK);
    CHECK(quantize_projgrad(g, q2, 255, &c) == MEZO_OK);
    CHECK(memcmp(q, q2, 255) == 0);
    for (a = 0; a < 3; ++a) {
        int qmax;
        c.kind = MEZO_CODEC_SIGNED_LOG;
        c.alpha = alphas[a];
        qmax = alphas[a] == 1.0f ? 88 : 127;  /* the natural log's codes stop at 88 */
        for (i = 0; i < 2 * qmax + 1; ++i) q[i] = (int8_t)(i - qmax);
        CHECK(mezo_dequantize(q, g, (uint32_t)(2 * qmax + 1), &c) == MEZO_OK);
        CHECK(quantize_projgrad(g, q2, (uint32_t)(2 * qmax + 1), &c) == MEZO_OK);
        CHECK(memcmp(q, q2, (size_t)(2 * qmax + 1)) == 0);
        q[0] = (int8_t)(qmax == 127 ? -128 : qmax + 1);
        CHECK(mezo_dequantize(q, g, 1, &c) == MEZO_ERANGE);
    }
    c.kind = MEZO_CODEC_LINEAR;
    g[0] = NAN;
    CHECK(quantize_projgrad(g, q2, 1, &c) == MEZO_ERANGE);
    c.scale = 0.0f;
    CHECK(quantize_projgrad(g, q2, 1, &c) == MEZO_ERANGE);
    c.kind = 7;
    CHECK(quantize_projgrad(g, q2, 1, &c) == MEZO_ERANGE);
    CHECK(quantize_projgrad(g, q2, 1, NULL) == MEZO_EINVAL);
    c.kind = MEZO_CODEC_LINEAR;
    c.scale = 1.0f;
    CHECK(quantize_projgrad(NULL, NULL, 0, &c) == MEZO_OK);
}

/* the coefficient the host forms for code q: fl32(-lr * q * scale), times
 * sqrt(2 ln 2) for the fast Gaussian (rounded once more to fp32) */
static float coef_of(int q, float lr, float scale, int fast)
{
    const float deq = (float)((double)q * (double)scale);
    const float c = (float)(-(double)lr * (double)deq);
    return fast ? (float)((double)c * 1.17741002251547469101) : c;
}

static void check_update_records(void)
{
    mezo_paramset_t ps;
    mezo_codec_t c = {MEZO_CODEC_LINEAR, 1.0f / 127.0f, 0.0f};
    mezo_seed_t s[6];
    int8_t q[6] = {3, 0, -5, 0, 127, -1};
    const float lr = 1e-3f;
    unsigned long before;
    uint32_t n, i, k;
    CHECK(create1(T(0x100000, 5000, 0, MEZO_F32, 0, 0), &ps) == MEZO_OK);
    for (i = 0; i < 6; ++i) s[i] = S(i / 2, 0, i % 2);
    /* argument checks first */
    CHECK(mezo_update_multi(NULL, s, q, 6, &c, lr, NULL) == MEZO_EINVAL);
    CHECK(mezo_update_multi(ps, NULL, q, 6, &c, lr, NULL) == MEZO_EINVAL);
    CHECK(mezo_update_multi(ps, s, q, 6, NULL, lr, NULL) == MEZO_EINVAL);
    CHECK(mezo_update_multi(ps, s, q, 6, &c, NAN, NULL) == MEZO_ERANGE);
    q[2] = -128;
    CHECK(mezo_update_multi(ps, s, q, 6, &c, lr, NULL) == MEZO_ERANGE);
    q[2] = -5;
    s[3] = S(0, 0, 1);  /* equal to s[1] */
    CHECK(mezo_update_multi(ps, s, q, 6, &c, lr, NULL) == MEZO_EORDER);
    s[3] = S(1, 0, 1);
    before = double_engine_launches(MEZO_F32);
    CHECK(mezo_update_multi(ps, s, q, 0, &c, lr, NULL) == MEZO_OK);
    CHECK(mezo_update_multi(ps, s, q, 6, &c, 0.0f, NULL) == MEZO_OK);
    CHECK(double_engine_launches(MEZO_F32) == before);
    /* zero codes dropped, the rest in order, the last flagged */
    CHECK(mezo_update_multi(ps, s, q, 6, &c, lr, NULL) == MEZO_OK);
    CHECK(double_engine_launches(MEZO_F32) == before + 1);
    n = double_last_records(g_coef, g_last, g_mach, MAXREC);
    CHECK(n == 4);
    for (i = 0, k = 0; i < 6; ++i) {
        if (q[i] == 0) continue;
        CHECK(g_coef[k] == coef_of(q[i], lr, c.scale, 1));
        CHECK(g_mach[k] == (uint32_t)s[i].machine);
        CHECK(g_last[k] == (k + 1 == n));
        ++k;
    }
    /* the portable Gaussian takes the coefficient itself */
    CHECK(mezo_paramset_set_gaussian(ps, MEZO_GAUSS_PORTABLE) == MEZO_OK);
    CHECK(mezo_update_multi(ps, s, q, 6, &c, lr, NULL) == MEZO_OK);
    n = double_last_records(g_coef, g_last, g_mach, MAXREC);
    CHECK(n == 4 && g_coef[0] == coef_of(3, lr, c.scale, 0));
    CHECK(mezo_paramset_set_gaussian(ps, 2) == MEZO_EINVAL);
    CHECK(mezo_paramset_set_gaussian(ps, MEZO_GAUSS_FAST) == MEZO_OK);
    mezo_paramset_destroy(ps);
}

static void check_perturb_calls(void)
{
    mezo_paramset_t ps;
    mezo_seed_t s[3] = {{0, 0, 0}, {0, 0, 1}, {1, 0, 0}};
    float sc[3] = {1e-3f, 0.0f, -2e-3f};
    uint32_t n;
    CHECK(create1(T(0x100000, 4096, 7, MEZO_BF16, 0, 0), &ps) == MEZO_OK);
    CHECK(mezo_perturb(ps, s[0], INFINITY, NULL) == MEZO_ERANGE);
    CHECK(mezo_perturb(NULL, s[0], 1.0f, NULL) == MEZO_EINVAL);
    CHECK(mezo_perturb(ps, s[0], 0.0f, NULL) == MEZO_OK);
    CHECK(mezo_perturb(ps, s[0], 1e-3f, NULL) == MEZO_OK);
    n = double_last_records(g_coef, g_last, g_mach, MAXREC);
    CHECK(n == 1 && g_last[0] == 1);
    /* several perturbations, each its own step; zero scales dropped */
    CHECK(mezo_perturb_multi(ps, s, sc, 3, NULL) == MEZO_OK);
    n = double_last_records(g_coef, g_last, g_mach, MAXREC);
    CHECK(n == 2 && g_last[0] == 1 && g_last[1] == 1 && g_mach[1] == 1);
    sc[1] = NAN;
    CHECK(mezo_perturb_multi(ps, s, sc, 3, NULL) == MEZO_ERANGE);
    CHECK(mezo_perturb_multi(ps, NULL, sc, 3, NULL) == MEZO_EINVAL);
    CHECK(mezo_perturb_multi(ps, NULL, NULL, 0, NULL) == MEZO_OK);
    mezo_paramset_destroy(ps);
}

static mezo_seed_t* seeds_n(uint32_t n, uint32_t step)
{
    mezo_seed_t* s = (mezo_seed_t*)malloc(n * sizeof(mezo_seed_t));
    uint32_t i;
    for (i = 0; i < n; ++i) s[i] = S(i, step, 0);
    return s;
}

static int8_t* codes_n(uint32_t n, int zero_every)
{
    int8_t* q = (int8_t*)malloc(n);
    uint32_t i;
    for (i = 0; i < n; ++i) q[i] = (int8_t)(zero_every && i % (uint32_t)zero_every == 0 ? 0 : 1 + (int)(i % 126));
    return q;
}

static void check_staging_and_replay(void)
{
    mezo_paramset_t ps;
    mezo_codec_t c = {MEZO_CODEC_LINEAR, 1.0f / 127.0f, 0.0f};
    const uint32_t sizes[6] = {40, 40, 300, 33, 5000, 40};
    mezo_seed_t* s = seeds_n(70000, 0);
    int8_t* q = codes_n(70000, 0);
    mezo_step_t st[4];
    unsigned long before, syncs;
    uint32_t n, i, r;
    CHECK(create1(T(0x100000, 3000, 0, MEZO_F32, 0, 0), &ps) == MEZO_OK);
    /* staged lists (> 32 records) cycle through the slot ring and grow it */
    for (r = 0; r < 3; ++r)
        for (i = 0; i < 6; ++i) {
            CHECK(mezo_update_multi(ps, s, q, sizes[i], &c, 1e-4f, NULL) == MEZO_OK);
            n = double_last_records(g_coef, g_last, g_mach, MAXREC);
            CHECK(n == sizes[i] && g_mach[n - 1] == n - 1 && g_last[n - 1] == 1 && g_last[0] == (n == 1));
        }
    /* a replay: each step's last kept record is flagged; empty, all-zero and
     * zero-lr steps add nothing */
    {
        int8_t* z = codes_n(3, 1);  /* all zero */
        mezo_seed_t* s1 = seeds_n(3, 1);
        mezo_seed_t* s2 = seeds_n(5, 2);
        st[0].seeds = s;
        st[0].q = q;
        st[0].K = 2;
        st[0].lr = 1e-3f;
        st[1].seeds = s1;
        st[1].q = z;
        st[1].K = 3;
        st[1].lr = 1e-3f;
        st[2].seeds = s2;
        st[2].q = q;
        st[2].K = 5;
        st[2].lr = 0.0f;
        st[3].seeds = s2;
        st[3].q = q;
        st[3].K = 5;
        st[3].lr = 1e-3f;
        CHECK(mezo_replay(ps, st, 4, &c, NULL) == MEZO_OK);
        n = double_last_records(g_coef, g_last, g_mach, MAXREC);
        CHECK(n == 7 && g_last[1] == 1 && g_last[0] == 0 && g_last[6] == 1 && g_last[5] == 0);
        st[1].seeds = s2;  /* unsorted across steps is fine; within a step it is not */
        s2[4] = S(0, 2, 0);
        CHECK(mezo_replay(ps, st, 4, &c, NULL) == MEZO_EORDER);
        CHECK(mezo_replay(ps, st, 0, &c, NULL) == MEZO_OK);
        CHECK(mezo_replay(ps, NULL, 2, &c, NULL) == MEZO_EINVAL);
        free(z);
        free(s1);
        free(s2);
    }
    /* a log longer than one launch's records runs as launches split at step
     * ends; a single longer step runs alone */
    before = double_engine_launches(MEZO_F32);
    for (i = 0; i < 3; ++i) {
        st[i].seeds = s;
        st[i].q = q;
        st[i].K = 30000;
        st[i].lr = 1e-4f;
    }
    CHECK(mezo_replay(ps, st, 3, &c, NULL) == MEZO_OK);
    CHECK(double_engine_launches(MEZO_F32) == before + 2);
    CHECK(double_last_records(g_coef, g_last, g_mach, MAXREC) == 30000);
    st[0].K = 70000;
    CHECK(mezo_replay(ps, st, 1, &c, NULL) == MEZO_OK);
    CHECK(double_last_records(g_coef, g_last, g_mach, MAXREC) == 70000);
    /* more than 2^32 - 1 terms: rejected from the step counts alone */
    st[0].K = 1u << 31;
    st[1].K = 1u << 31;
    CHECK(mezo_replay(ps, st, 2, &c, NULL) == MEZO_ERANGE);
    /* the slots' events are waited for before a slot is reused */
    syncs = double_event_syncs();
    for (i = 0; i < 9; ++i) CHECK(mezo_update_multi(ps, s, q, 64, &c, 1e-4f, NULL) == MEZO_OK);
    CHECK(double_event_syncs() >= syncs + 8);
    mezo_paramset_destroy(ps);
    free(s);
    free(q);
}

static float g_coef2[MAXREC];
static uint32_t g_last2[MAXREC], g_mach2[MAXREC];

/* mezo_replay_noalloc: the records mezo_replay would launch, through the
 * staging array, with no allocation and no event created */
static void check_replay_noalloc(void)
{
    mezo_paramset_t ps, fresh;
    mezo_codec_t c = {MEZO_CODEC_LINEAR, 1.0f / 127.0f, 0.0f};
    mezo_seed_t* s = seeds_n(70000, 0);
    int8_t* q = codes_n(70000, 5);  /* every 5th code zero: dropped */
    mezo_step_t st[3];
    unsigned long allocs, stages, launches;
    uint32_t n, n2, i;
    CHECK(create1(T(0x100000, 3000, 0, MEZO_BF16, 0, 0), &ps) == MEZO_OK);
    CHECK(create1(T(0x200000, 300, 1, MEZO_F32, 0, 0), &fresh) == MEZO_OK);
    for (i = 0; i < 3; ++i) {
        st[i].seeds = s;
        st[i].q = q;
        st[i].K = 400 + 37 * i;
        st[i].lr = 1e-3f;
    }
    /* no device tables yet: refused (creating them would allocate) */
    CHECK(mezo_replay_noalloc(fresh, st, 3, &c, NULL) == MEZO_EINVAL);
    CHECK(strlen(mezo_last_error()) > 0);
    CHECK(mezo_replay_noalloc(NULL, st, 3, &c, NULL) == MEZO_EINVAL);
    CHECK(mezo_replay_noalloc(ps, st, 3, NULL, NULL) == MEZO_EINVAL);
    CHECK(mezo_replay_noalloc(ps, st, 0, &c, NULL) == MEZO_OK);
    CHECK(mezo_replay(ps, st, 3, &c, NULL) == MEZO_OK);  /* creates the tables */
    n = double_last_records(g_coef, g_last, g_mach, MAXREC);
    allocs = double_allocation_calls();
    stages = double_stage_launches();
    launches = double_engine_launches(MEZO_BF16);
    for (i = 0; i < 20; ++i)  /* 20 streams: more than the tracked ones */
        CHECK(mezo_replay_noalloc(ps, st, 3, &c, (void*)(uintptr_t)(0x1000 * (i + 1))) == MEZO_OK);
    n2 = double_last_records(g_coef2, g_last2, g_mach2, MAXREC);
    CHECK(double_allocation_calls() == allocs);
    CHECK(double_engine_launches(MEZO_BF16) == launches + 20);
    CHECK(double_stage_launches() == stages + 20 * ((n + 31) / 32));
    CHECK(n2 == n && memcmp(g_coef, g_coef2, n * sizeof(float)) == 0 &&
          memcmp(g_last, g_last2, n * sizeof(uint32_t)) == 0 && memcmp(g_mach, g_mach2, n * sizeof(uint32_t)) == 0);
    /* a second, smaller call: only its own records are read */
    st[0].K = 40;
    CHECK(mezo_replay(ps, st, 1, &c, NULL) == MEZO_OK);
    n = double_last_records(g_coef, g_last, g_mach, MAXREC);
    CHECK(mezo_replay_noalloc(ps, st, 1, &c, NULL) == MEZO_OK);
    n2 = double_last_records(g_coef2, g_last2, g_mach2, MAXREC);
    CHECK(n == 32 && n2 == n && memcmp(g_coef, g_coef2, n * sizeof(float)) == 0);
    /* at most 32 records travel in the engine's arguments: no staging */
    stages = double_stage_launches();
    st[0].K = 20;
    CHECK(mezo_replay_noalloc(ps, st, 1, &c, NULL) == MEZO_OK);
    CHECK(double_stage_launches() == stages);
    /* argument checks as for mezo_replay, before anything is enqueued */
    q[3] = -128;
    CHECK(mezo_replay_noalloc(ps, st, 1, &c, NULL) == MEZO_ERANGE);
    q[3] = 4;
    st[0].lr = NAN;
    CHECK(mezo_replay_noalloc(ps, st, 1, &c, NULL) == MEZO_ERANGE);
    st[0].lr = 1e-3f;
    s[7] = S(3, 0, 0);
    CHECK(mezo_replay_noalloc(ps, st, 1, &c, NULL) == MEZO_EORDER);
    s[7] = S(7, 0, 0);
    /* more records than the staging array holds: refused; exactly 65536 fits */
    for (i = 0; i < 70000; ++i) q[i] = 1;
    st[0].K = 65537;
    CHECK(mezo_replay_noalloc(ps, st, 1, &c, NULL) == MEZO_ERANGE);
    st[0].K = 65536;
    CHECK(mezo_replay_noalloc(ps, st, 1, &c, NULL) == MEZO_OK);
    CHECK(double_last_records(g_coef, g_last, g_mach, MAXREC) == 65536 && g_last[65535] == 1 && g_last[65534] == 0);
    /* graph capture: every step is a kernel launch, so it may be captured */
    double_set_capturing(1);
    CHECK(mezo_replay_noalloc(ps, st, 1, &c, NULL) == MEZO_OK);
    double_set_capturing(0);
    /* the device its tables live on */
    double_set_device(2);
    CHECK(mezo_replay_noalloc(ps, st, 1, &c, NULL) == MEZO_EINVAL);
    double_set_device(0);
    mezo_paramset_destroy(fresh);
    mezo_paramset_destroy(ps);
    free(s);
    free(q);
}

static void check_streams_devices_capture(void)
{
    mezo_paramset_t ps, fresh;
    mezo_codec_t c = {MEZO_CODEC_LINEAR, 1.0f / 127.0f, 0.0f};
    mezo_seed_t* s = seeds_n(64, 0);
    int8_t* q = codes_n(64, 0);
    unsigned long syncs;
    uint64_t out[2];
    uintptr_t k;
    CHECK(create1(T(0x100000, 3000, 0, MEZO_F32, 0, 0), &ps) == MEZO_OK);
    /* 20 streams: the 17th and later take over the entry used longest ago */
    for (k = 1; k <= 16; ++k) CHECK(mezo_perturb(ps, S(0, 0, 0), 1e-3f, (void*)(k * 0x100)) == MEZO_OK);
    syncs = double_event_syncs();
    for (k = 17; k <= 20; ++k) CHECK(mezo_perturb(ps, S(0, 0, 0), 1e-3f, (void*)(k * 0x100)) == MEZO_OK);
    CHECK(double_event_syncs() == syncs + 4);
    /* a paramset stays on the device it was first used on */
    double_set_device(1);
    CHECK(mezo_perturb(ps, S(0, 0, 0), 1e-3f, NULL) == MEZO_EINVAL);
    CHECK(strlen(mezo_last_error()) > 0);
    double_set_device(0);
    /* graph capture: no first use (it allocates), no staged list */
    CHECK(create1(T(0x200000, 100, 0, MEZO_F32, 0, 0), &fresh) == MEZO_OK);
    double_set_capturing(1);
    CHECK(mezo_perturb(fresh, S(0, 0, 0), 1e-3f, NULL) == MEZO_EINVAL);
    CHECK(mezo_perturb(ps, S(0, 0, 0), 1e-3f, NULL) == MEZO_OK);
    CHECK(mezo_update_multi(ps, s, q, 32, &c, 1e-4f, NULL) == MEZO_OK);
    CHECK(mezo_update_multi(ps, s, q, 33, &c, 1e-4f, NULL) == MEZO_EINVAL);
    CHECK(mezo_checksum(ps, out, NULL) == MEZO_OK);
    CHECK(mezo_checksum(fresh, out, NULL) == MEZO_EINVAL);
    double_set_capturing(0);
    CHECK(mezo_checksum(ps, (uint64_t*)((char*)out + 4), NULL) == MEZO_EINVAL);
    CHECK(mezo_checksum(NULL, out, NULL) == MEZO_EINVAL);
    /* a device allocation that fails: the call reports it, frees what it
     * made, and a later call starts over */
    double_fail_malloc_in(1);
    CHECK(mezo_perturb(fresh, S(0, 0, 0), 1e-3f, NULL) == MEZO_EHIP);
    CHECK(strlen(mezo_last_error()) > 0);
    CHECK(mezo_perturb(fresh, S(0, 0, 0), 1e-3f, NULL) == MEZO_OK);
    mezo_paramset_destroy(fresh);
    mezo_paramset_destroy(ps);
    free(s);
    free(q);
}

static void check_from_mixed_checksum_nf4(void)
{
    mezo_paramset_t dst, src, bad, overlap, mixed;
    mezo_tensor_t t[3];
    mezo_codec_t c = {MEZO_CODEC_LINEAR, 1.0f / 127.0f, 0.0f};
    mezo_seed_t s[2] = {{0, 0, 0}, {1, 0, 0}};
    int8_t q[2] = {3, 4};
    unsigned long f, b, n4, ck, nf;
    uint64_t out;
    t[0] = T(0x100000, 1024, 0, MEZO_F32, 0, 0);
    t[1] = T(0x200000, 512, 1, MEZO_BF16, 0, 0);
    CHECK(mezo_paramset_create(t, 2, &dst) == MEZO_OK);
    t[0].data = (void*)0x300000;
    t[1].data = (void*)0x400000;
    CHECK(mezo_paramset_create(t, 2, &src) == MEZO_OK);
    t[0].numel = 1000;
    CHECK(mezo_paramset_create(t, 2, &bad) == MEZO_OK);
    t[0] = T(0x100800, 1024, 0, MEZO_F32, 0, 0);
    CHECK(mezo_paramset_create(t, 2, &overlap) == MEZO_OK);
    CHECK(mezo_update_multi_from(dst, bad, s, q, 2, &c, 1e-3f, NULL) == MEZO_EINVAL);
    CHECK(mezo_perturb_from(dst, overlap, s[0], 1e-3f, NULL) == MEZO_EOVERLAP);
    CHECK(mezo_update_multi_from(dst, src, s, q, 2, &c, NAN, NULL) == MEZO_ERANGE);
    f = double_engine_launches(MEZO_F32);
    b = double_engine_launches(MEZO_BF16);
    CHECK(mezo_update_multi_from(dst, src, s, q, 2, &c, 1e-3f, NULL) == MEZO_OK);
    CHECK(double_last_out_of_place());
    /* nothing to apply out of place is still a copy */
    CHECK(mezo_perturb_from(dst, src, s[0], 0.0f, NULL) == MEZO_OK);
    CHECK(double_engine_launches(MEZO_F32) == f + 2 && double_engine_launches(MEZO_BF16) == b + 2);
    /* the identical set means in place */
    CHECK(mezo_perturb_from(dst, dst, s[0], 1e-3f, NULL) == MEZO_OK);
    CHECK(!double_last_out_of_place());
    /* one launch per storage type present */
    t[0] = T(0x500000, 100, 0, MEZO_F32, 0, 0);
    t[1] = T(0x600000, 70001, 1, MEZO_NF4, 0x700000, 0);
    t[2] = T(0x800000, 5000, 2, MEZO_BF16, 0, 0);
    CHECK(mezo_paramset_create(t, 3, &mixed) == MEZO_OK);
    f = double_engine_launches(MEZO_F32);
    b = double_engine_launches(MEZO_BF16);
    n4 = double_engine_launches(MEZO_NF4);
    CHECK(mezo_update_multi(mixed, s, q, 2, &c, 1e-3f, NULL) == MEZO_OK);
    CHECK(double_engine_launches(MEZO_F32) == f + 1 && double_engine_launches(MEZO_BF16) == b + 1 &&
          double_engine_launches(MEZO_NF4) == n4 + 1);
    ck = double_checksum_launches();
    CHECK(mezo_checksum(mixed, &out, NULL) == MEZO_OK);
    CHECK(double_checksum_launches() == ck + 1);
    /* the standalone NF4 conversions */
    nf = double_nf4_launches();
    CHECK(mezo_nf4_quantize((void*)0x1000, 9, 64, (void*)0x2000, (float*)0x3000, NULL) == MEZO_EDTYPE);
    CHECK(mezo_nf4_quantize((void*)0x1000, MEZO_F32, 64, (void*)0x1080, (float*)0x3000, NULL) == MEZO_EOVERLAP);
    CHECK(mezo_nf4_dequantize((void*)0x2000, (float*)0x2010, 64, (void*)0x1000, MEZO_F32, NULL) == MEZO_EOVERLAP);
    CHECK(mezo_nf4_quantize((void*)0x1000, MEZO_BF16, 64, (void*)0x2000, (float*)0x3000, NULL) == MEZO_OK);
    CHECK(mezo_nf4_dequantize((void*)0x2000, (float*)0x3000, 64, (void*)0x1000, MEZO_F32, NULL) == MEZO_OK);
    CHECK(double_nf4_launches() == nf + 2);
    mezo_paramset_destroy(mixed);
    mezo_paramset_destroy(overlap);
    mezo_paramset_destroy(bad);
    mezo_paramset_destroy(src);
    mezo_paramset_destroy(dst);
}

static void check_inspection_and_messages(void)
{
    unsigned long g = double_generate_launches();
    int code;
    CHECK(mezo_debug_generate(S(0, 0, 0), 0, MEZO_MAX_NUMEL - 4, 8, 0, (uint32_t*)0x1000, NULL, NULL) ==
          MEZO_EINVAL);
    CHECK(mezo_debug_generate(S(0, 0, 0), 0, 0, 16, 7, (uint32_t*)0x1000, NULL, NULL) == MEZO_EINVAL);
    CHECK(mezo_debug_generate(S(0, 0, 0), 0, 0, 0, 0, (uint32_t*)0x1000, NULL, NULL) == MEZO_OK);
    CHECK(mezo_debug_generate(S(0, 0, 0), 0, 3, 1000, 0, (uint32_t*)0x1000, NULL, NULL) == MEZO_OK);
    CHECK(mezo_debug_box_muller((const uint32_t*)0x1008, 4, 0, (float*)0x2000, NULL) == MEZO_EINVAL);
    CHECK(mezo_debug_box_muller((const uint32_t*)0x1000, 4, 0, (float*)0x2000, NULL) == MEZO_OK);
    CHECK(double_generate_launches() == g + 2);
    for (code = MEZO_ENOMEM; code <= MEZO_OK; ++code) CHECK(strcmp(mezo_strerror(code), "unknown error code") != 0);
    CHECK(strcmp(mezo_strerror(-99), "unknown error code") == 0);
    CHECK(mezo_version() > 0);
}

/* four callers at once, each on its own paramset and stream */
static void* worker(void* arg)
{
    const uintptr_t id = (uintptr_t)arg;
    mezo_paramset_t ps;
    mezo_codec_t c = {MEZO_CODEC_LINEAR, 1.0f / 127.0f, 0.0f};
    mezo_seed_t* s = seeds_n(100, 0);
    int8_t* q = codes_n(100, 7);
    int i, bad = 0;
    if (create1(T(0x1000000 * (id + 1), 20000, (uint32_t)id, MEZO_BF16, 0, 0), &ps) != MEZO_OK) return (void*)1;
    for (i = 0; i < 200; ++i) {
        bad |= mezo_update_multi(ps, s, q, (uint32_t)(1 + (i * 7) % 100), &c, 1e-4f, (void*)(id * 0x10)) != MEZO_OK;
        bad |= mezo_perturb(ps, S(id, (uint32_t)i, 0), 1e-3f, (void*)(id * 0x10)) != MEZO_OK;
    }
    mezo_paramset_destroy(ps);
    free(s);
    free(q);
    return (void*)(uintptr_t)bad;
}

static void check_threads(void)
{
    pthread_t th[4];
    uintptr_t i;
    for (i = 0; i < 4; ++i) pthread_create(&th[i], NULL, worker, (void*)i);
    for (i = 0; i < 4; ++i) {
        void* r = NULL;
        pthread_join(th[i], &r);
        CHECK(r == NULL);
    }
}

int main(void)
{
    check_create();
    check_codec();
    check_update_records();
    check_perturb_calls();
    check_staging_and_replay();
    check_streams_devices_capture();
    check_replay_noalloc();
    check_from_mixed_checksum_nf4();
    check_inspection_and_messages();
    check_threads();
    /* every paramset destroyed: no table, staging slot or event is left */
    CHECK(double_device_allocations() == 0);
    CHECK(double_events_live() == 0);
    printf("abi_host_check: %d checks, %d failed\n", g_checks, g_failed);
    return g_failed ? 1 : 0;
}
