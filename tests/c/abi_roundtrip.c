/*
 * abi_roundtrip.c — the engine driven from plain C through include/mezo.h
 * alone (no Python, no torch): device memory from the HIP runtime's C API,
 * one fp32 and one bf16 tensor, a perturb (Algorithm 1, PerturbParameters), a
 * fused 4-seed update (the apply loop), a 3-step replay (Appendix B), an
 * update with the portable Gaussian (bit-exact) and a checksum
 * (ChecksumMatch), each compared with the CPU oracle (test infrastructure,
 * linked here only). Exit status 0 when every check passes.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "mezo.h"
#include "mezo_oracle.h"

#define CHECK(cond, ...)                                    \
    do {                                                    \
        if (!(cond)) {                                      \
            fprintf(stderr, "FAIL: " __VA_ARGS__);          \
            fprintf(stderr, "\n");                          \
            return 1;                                       \
        }                                                   \
    } while (0)

static uint16_t to_bf16_rne(float x)
{
    uint32_t u;
    memcpy(&u, &x, 4);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

static double bf16_value(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

int main(void)
{
    enum { NF = 100003, NB = 4097, K = 4 };
    float* hf = malloc(NF * sizeof(float));
    uint16_t* hb = malloc(NB * sizeof(uint16_t));
    float* rf = malloc(NF * sizeof(float));
    uint16_t* rb = malloc(NB * sizeof(uint16_t));
    float* gf = malloc(NF * sizeof(float));
    uint16_t* gb = malloc(NB * sizeof(uint16_t));
    CHECK(hf && hb && rf && rb && gf && gb, "host allocation");
    /* seeded inputs: a fixed pattern of magnitude ~0.02 */
    for (int i = 0; i < NF; ++i) hf[i] = 0.02f * sinf(0.001f * (float)i + 0.3f);
    for (int i = 0; i < NB; ++i) hb[i] = to_bf16_rne(0.02f * cosf(0.002f * (float)i));

    void *df = NULL, *db = NULL;
    uint64_t* dsum = NULL;
    CHECK(hipSetDevice(0) == hipSuccess, "hipSetDevice");
    CHECK(hipMalloc(&df, NF * sizeof(float)) == hipSuccess, "hipMalloc");
    CHECK(hipMalloc(&db, NB * sizeof(uint16_t)) == hipSuccess, "hipMalloc");
    CHECK(hipMalloc((void**)&dsum, sizeof(uint64_t)) == hipSuccess, "hipMalloc");
    CHECK(hipMemcpy(df, hf, NF * sizeof(float), hipMemcpyHostToDevice) == hipSuccess, "copy");
    CHECK(hipMemcpy(db, hb, NB * sizeof(uint16_t), hipMemcpyHostToDevice) == hipSuccess, "copy");

    mezo_tensor_t t[2];
    memset(t, 0, sizeof(t));
    t[0].data = df; t[0].numel = NF; t[0].tensor_id = 7; t[0].dtype = MEZO_F32;
    t[1].data = db; t[1].numel = NB; t[1].tensor_id = 2; t[1].dtype = MEZO_BF16;
    mezo_paramset_t ps = NULL;
    CHECK(mezo_paramset_create(t, 2, &ps) == MEZO_OK, "create");

    orc_seed_t os = {42u, 3u, 1u};
    orc_seed_t oseeds[K] = {{0u, 5u, 0u}, {1u, 5u, 0u}, {2u, 5u, 0u}, {3u, 5u, 0u}};
    mezo_seed_t s = {42u, 3u, 1u};
    mezo_seed_t seeds[K] = {{0u, 5u, 0u}, {1u, 5u, 0u}, {2u, 5u, 0u}, {3u, 5u, 0u}};
    int8_t q[K] = {17, -90, 127, -3};
    mezo_codec_t codec = {MEZO_CODEC_LINEAR, 1.0f / 127.0f, 1.0f};
    /* a log of T steps of K seeds each, packed step after step */
    enum { T = 3 };
    orc_seed_t olog[T * K];
    mezo_seed_t mlog[T * K];
    int8_t qlog[T * K];
    uint32_t klog[T];
    float lrlog[T];
    mezo_step_t steps[T];
    for (int t = 0; t < T; ++t) {
        for (int k = 0; k < K; ++k) {
            const int i = t * K + k;
            olog[i].machine = mlog[i].machine = (uint64_t)k;
            olog[i].step = mlog[i].step = 10u + (uint32_t)t;
            olog[i].sample = mlog[i].sample = 0u;
            qlog[i] = (int8_t)(((t * 37 + k * 53) % 255) - 127);
        }
        klog[t] = K;
        lrlog[t] = 1e-3f * (float)(t + 1);
        steps[t].seeds = mlog + t * K;
        steps[t].q = qlog + t * K;
        steps[t].K = K;
        steps[t].lr = lrlog[t];
    }

    for (int step = 0; step < 4; ++step) {
        /* the oracle starts from what the GPU holds before the step */
        CHECK(hipMemcpy(rf, df, NF * sizeof(float), hipMemcpyDeviceToHost) == hipSuccess, "copy back");
        CHECK(hipMemcpy(rb, db, NB * sizeof(uint16_t), hipMemcpyDeviceToHost) == hipSuccess, "copy back");
        memcpy(hb, rb, NB * sizeof(uint16_t));  /* the step's bf16 input */
        if (step == 0) {
            CHECK(mezo_perturb(ps, s, 1e-3f, NULL) == MEZO_OK, "perturb");
            CHECK(orc_perturb(rf, ORC_F32, 7u, NULL, 0, NF, os, 1e-3f) == 0, "oracle perturb");
            CHECK(orc_perturb(rb, ORC_BF16, 2u, NULL, 0, NB, os, 1e-3f) == 0, "oracle perturb");
        } else if (step == 1) {
            CHECK(mezo_update_multi(ps, seeds, q, K, &codec, 1e-3f, NULL) == MEZO_OK, "update");
            CHECK(orc_update(rf, ORC_F32, 7u, NULL, 0, NF, oseeds, q, K, ORC_CODEC_LINEAR, 1.0f / 127.0f,
                             1.0f, 1e-3f) == 0, "oracle update");
            CHECK(orc_update(rb, ORC_BF16, 2u, NULL, 0, NB, oseeds, q, K, ORC_CODEC_LINEAR, 1.0f / 127.0f,
                             1.0f, 1e-3f) == 0, "oracle update");
        } else if (step == 2) {
            CHECK(mezo_replay(ps, steps, T, &codec, NULL) == MEZO_OK, "replay");
            CHECK(orc_replay(rf, ORC_F32, 7u, NULL, 0, NF, olog, qlog, klog, lrlog, T, ORC_CODEC_LINEAR,
                             1.0f / 127.0f, 1.0f) == 0, "oracle replay");
            CHECK(orc_replay(rb, ORC_BF16, 2u, NULL, 0, NB, olog, qlog, klog, lrlog, T, ORC_CODEC_LINEAR,
                             1.0f / 127.0f, 1.0f) == 0, "oracle replay");
        } else {
            CHECK(mezo_paramset_set_gaussian(ps, MEZO_GAUSS_PORTABLE) == MEZO_OK, "set_gaussian");
            CHECK(mezo_update_multi(ps, seeds, q, K, &codec, 1e-3f, NULL) == MEZO_OK, "portable update");
            CHECK(orc_update_portable(rf, ORC_F32, 7u, NULL, 0, NF, oseeds, q, K, ORC_CODEC_LINEAR,
                                      1.0f / 127.0f, 1.0f, 1e-3f) == 0, "oracle portable update");
            CHECK(orc_update_portable(rb, ORC_BF16, 2u, NULL, 0, NB, oseeds, q, K, ORC_CODEC_LINEAR,
                                      1.0f / 127.0f, 1.0f, 1e-3f) == 0, "oracle portable update");
        }
        CHECK(hipDeviceSynchronize() == hipSuccess, "sync");
        CHECK(hipMemcpy(gf, df, NF * sizeof(float), hipMemcpyDeviceToHost) == hipSuccess, "copy back");
        CHECK(hipMemcpy(gb, db, NB * sizeof(uint16_t), hipMemcpyDeviceToHost) == hipSuccess, "copy back");
        if (step == 3) {
            /* the portable Gaussian: every bit */
            CHECK(memcmp(gf, rf, NF * sizeof(float)) == 0, "portable update: fp32 not bit-exact");
            CHECK(memcmp(gb, rb, NB * sizeof(uint16_t)) == 0, "portable update: bf16 not bit-exact");
            printf("step 3 ok: portable update bit-exact\n");
            continue;
        }
        /* fp32: max |diff| <= 1e-6 max |ref| */
        double scale = 0.0, err = 0.0;
        for (int i = 0; i < NF; ++i) {
            scale = fmax(scale, fabs((double)rf[i]));
            err = fmax(err, fabs((double)gf[i] - (double)rf[i]));
        }
        CHECK(err <= 1e-6 * scale, "step %d: fp32 max abs error %.3e > %.3e", step, err, 1e-6 * scale);
        /* bf16: one ulp of the larger of the operation's input and the result */
        int far = 0;
        for (int i = 0; i < NB; ++i) {
            double g = bf16_value(gb[i]), r = bf16_value(rb[i]);
            double m = fmax(fabs(r), fabs(bf16_value(hb[i])));
            double ulp = m > 0 ? ldexp(1.0, (int)floor(log2(m)) - 7) : ldexp(1.0, -133);
            if (fabs(g - r) > ulp) ++far;
        }
        CHECK(far == 0, "step %d: %d bf16 elements off by more than one ulp", step, far);
        printf("step %d ok: fp32 max abs error %.3e (bar %.3e)\n", step, err, 1e-6 * scale);
    }

    /* ChecksumMatch of what the GPU holds, by the oracle's definition */
    uint64_t sum = 0;
    CHECK(mezo_checksum(ps, dsum, NULL) == MEZO_OK, "checksum");
    CHECK(hipMemcpy(&sum, dsum, sizeof(sum), hipMemcpyDeviceToHost) == hipSuccess, "copy back");
    uint64_t want = orc_checksum(gf, NF * sizeof(float), 7u) + orc_checksum(gb, NB * sizeof(uint16_t), 2u);
    CHECK(sum == want, "checksum %016llx != %016llx", (unsigned long long)sum, (unsigned long long)want);

    mezo_paramset_destroy(ps);
    (void)hipFree(df);
    (void)hipFree(db);
    (void)hipFree(dsum);
    free(hf); free(hb); free(rf); free(rb); free(gf); free(gb);
    printf("abi_roundtrip ok: checksum %016llx\n", (unsigned long long)sum);
    return 0;
}
