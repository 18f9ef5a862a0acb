/*
 * mezo_oracle.c — CPU oracle for the seeded perturbation engine.
 *
 * TEST INFRASTRUCTURE ONLY: called by the tests, the smoke check and the
 * benchmark's CPU-baseline leg, never by the product path. Plain C99 with
 * optional OpenMP over independent elements; fp64 arithmetic; no fast-math,
 * no contraction (built with -ffp-contract=off), no flush of subnormals.
 * Every function states the passage of arXiv 2306.10015 it follows; the
 * header lists the readings taken where the paper is silent.
 */
#include "mezo_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <stdint.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------------ */
/* Philox4x32-10 (Salmon et al., SC'11, Section 4 / Table 2).               */
/* The paper only asks for an RNG that can be reset with a seed and that    */
/* regenerates the same noise on every machine (Algorithm 1,                */
/* PerturbParameters; Appendix B on cross-device determinism). A counter-   */
/* based generator gives each element its noise without a sequential walk.  */
/* ------------------------------------------------------------------------ */

/* The two round multipliers and the two key (Weyl) increments of Philox4x32. */
#define PHILOX_MUL_A 0xD2511F53u
#define PHILOX_MUL_B 0xCD9E8D57u
#define PHILOX_WEYL_A 0x9E3779B9u
#define PHILOX_WEYL_B 0xBB67AE85u

/* One Philox S-box round: two full 32x32->64 products, then a Feistel-like
 * mixing of the high halves with the other two words and the round key. */
static void philox_round(uint32_t x[4], const uint32_t k[2])
{
    uint64_t pa = (uint64_t)PHILOX_MUL_A * (uint64_t)x[0];
    uint64_t pb = (uint64_t)PHILOX_MUL_B * (uint64_t)x[2];
    uint32_t y0 = (uint32_t)(pb >> 32) ^ x[1] ^ k[0];
    uint32_t y1 = (uint32_t)pb;
    uint32_t y2 = (uint32_t)(pa >> 32) ^ x[3] ^ k[1];
    uint32_t y3 = (uint32_t)pa;
    x[0] = y0;
    x[1] = y1;
    x[2] = y2;
    x[3] = y3;
}

void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    uint32_t x[4] = {ctr[0], ctr[1], ctr[2], ctr[3]};
    uint32_t k[2] = {key[0], key[1]};
    for (int r = 0; r < 10; ++r) {
        if (r > 0) { /* key schedule: add the Weyl constants between rounds */
            k[0] += PHILOX_WEYL_A;
            k[1] += PHILOX_WEYL_B;
        }
        philox_round(x, k);
    }
    memcpy(out, x, sizeof(x));
}

/* Seed -> key and counter. The seed of Algorithm 1 is (self_time, t, sample
 * index); the key carries the 64-bit machine id, the counter carries the
 * element's block (4 elements per block), the tensor, the sample and the step,
 * so every parameter gets its own, position-fixed, draw. */
void orc_block_words(orc_seed_t s, uint32_t tensor_id, uint64_t e, uint32_t out[4])
{
    uint32_t ctr[4];
    uint32_t key[2];
    ctr[0] = (uint32_t)(e >> 2);
    ctr[1] = tensor_id;
    ctr[2] = s.sample;
    ctr[3] = s.step;
    key[0] = (uint32_t)(s.machine & 0xFFFFFFFFu);
    key[1] = (uint32_t)(s.machine >> 32);
    orc_philox4x32_10(ctr, key, out);
}

/* ------------------------------------------------------------------------ */
/* z ~ N(0,1) (Algorithm 1, PerturbParameters): Box-Muller (Box & Muller,   */
/* 1958) on uniforms built from the top 24 bits of each word, so that they  */
/* are exact in any binary floating-point format with >= 24-bit mantissa.   */
/*   u1 = ((w_a >> 8) + 1) / 2^24  in (0, 1]   (log argument never 0)       */
/*   u2 =  (w_b >> 8)      / 2^24  in [0, 1)                                */
/*   r = sqrt(-2 ln u1), phi = 2 pi u2, z = (r cos phi, r sin phi)          */
/* Words (w0, w1) give z[0], z[1]; words (w2, w3) give z[2], z[3].          */
/* ------------------------------------------------------------------------ */

static const double TWO_PI = 6.283185307179586476925286766559;

void orc_box_muller(const uint32_t w[4], double z[4])
{
    for (int p = 0; p < 2; ++p) {
        double u1 = (double)((w[2 * p] >> 8) + 1u) / 16777216.0;
        double u2 = (double)(w[2 * p + 1] >> 8) / 16777216.0;
        double r = sqrt(-2.0 * log(u1));
        double phi = TWO_PI * u2;
        z[2 * p] = r * cos(phi);
        z[2 * p + 1] = r * sin(phi);
    }
}

/* Box-Muller of n blocks of given words (4 per block), each z rounded once
 * to fp32 as orc_z does: for checking a transform over chosen inputs. */
void orc_box_muller_blocks(const uint32_t* w, uint64_t n_blocks, float* z)
{
    long long n = (long long)n_blocks;
#pragma omp parallel for schedule(static)
    for (long long b = 0; b < n; ++b) {
        double zz[4];
        orc_box_muller(w + 4 * b, zz);
        for (int j = 0; j < 4; ++j) z[4 * b + j] = (float)zz[j];
    }
}

float orc_z(orc_seed_t s, uint32_t tensor_id, uint64_t e)
{
    uint32_t w[4];
    double z[4];
    orc_block_words(s, tensor_id, e, w);
    orc_box_muller(w, z);
    return (float)z[e & 3u];
}

int orc_generate(orc_seed_t s, uint32_t tensor_id, uint64_t first, uint64_t count,
                 uint32_t* words, float* z)
{
    if (count > 0 && (first + count - 1) >> 34) return -1;
    long long n = (long long)count;
#pragma omp parallel for schedule(static)
    for (long long i = 0; i < n; ++i) {
        uint64_t e = first + (uint64_t)i;
        if (words) {
            uint32_t w[4];
            orc_block_words(s, tensor_id, e, w);
            words[i] = w[e & 3u];
        }
        if (z) z[i] = orc_z(s, tensor_id, e);
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Storage rounding: one round-to-nearest-even from the exact fp64 value     */
/* straight to the storage format (no double rounding through fp32 for bf16).*/
/* ------------------------------------------------------------------------ */

float orc_round_f32(double x)
{
    return (float)x; /* C conversion under the default rounding mode: RNE */
}

uint16_t orc_round_bf16(double x)
{
    uint16_t sign = signbit(x) ? 0x8000u : 0u;
    if (isnan(x)) return 0x7FC0u;
    double ax = fabs(x);
    if (ax == 0.0) return sign;
    if (isinf(ax)) return (uint16_t)(sign | 0x7F80u);
    /* ax = m * 2^ex with m in [0.5, 1): bf16 keeps 8 significant bits, so the
     * spacing of representable values around ax is 2^(ex-8); below the
     * smallest normal (2^-126) the spacing stays at 2^-133. */
    int ex;
    (void)frexp(ax, &ex);
    int sp = ex - 8;
    if (sp < -133) sp = -133;
    double q = rint(ldexp(ax, -sp)); /* exact scaling; rint ties to even */
    double r = ldexp(q, sp);
    if (r >= 0x1p128) return (uint16_t)(sign | 0x7F80u); /* overflow */
    float f = (float)r;                                  /* exact */
    uint32_t bits;
    memcpy(&bits, &f, sizeof(bits));
    return (uint16_t)(sign | (uint16_t)(bits >> 16));
}

static double bf16_to_double(uint16_t b)
{
    uint32_t bits = (uint32_t)b << 16;
    float f;
    memcpy(&f, &bits, sizeof(f));
    return (double)f;
}

static double load_theta(const void* theta, int dtype, uint64_t i)
{
    if (dtype == ORC_F32) return (double)((const float*)theta)[i];
    return bf16_to_double(((const uint16_t*)theta)[i]);
}

static void store_theta(void* theta, int dtype, uint64_t i, double v)
{
    if (dtype == ORC_F32)
        ((float*)theta)[i] = orc_round_f32(v);
    else
        ((uint16_t*)theta)[i] = orc_round_bf16(v);
}

/* ------------------------------------------------------------------------ */
/* One-byte projected gradient (Section 3: a signed log of the gradient,    */
/* clipped to +-127; the linear int8 code is the other                      */
/* codec the engine accepts). The range is the closed [-127, 127]; -128 is  */
/* never produced and rejected on input; rounding ties go to even.          */
/* ------------------------------------------------------------------------ */

/* Largest code magnitude of the signed-log code: the paper's clip at 127, or
 * less where a larger code would decode past fp32, i.e. fl32(exp(k/alpha) - 1)
 * would be infinite (alpha < ~1.4314; the natural log, alpha = 1: 88). The
 * default alpha = 1/ln 2 (a base-2 log) puts 127 just inside fp32. */
int orc_signed_log_qmax(float alpha)
{
    int k = 127;
    while (k > 0 && !isfinite((float)expm1((double)k / (double)alpha))) --k;
    return k;
}

static int codec_ok(int kind, float scale, float alpha)
{
    if (kind == ORC_CODEC_LINEAR) return isfinite(scale) && scale > 0.0f;
    if (kind == ORC_CODEC_SIGNED_LOG)
        return isfinite(alpha) && alpha > 0.0f && orc_signed_log_qmax(alpha) >= 1;
    return 0;
}

/* Largest |q| the codec produces and accepts. */
static int code_max(int kind, float alpha)
{
    return kind == ORC_CODEC_SIGNED_LOG ? orc_signed_log_qmax(alpha) : 127;
}

int orc_quantize(const float* g, int8_t* q, uint32_t n, int kind, float scale, float alpha)
{
    if (!codec_ok(kind, scale, alpha)) return -2;
    for (uint32_t i = 0; i < n; ++i)
        if (isnan(g[i])) return -2;
    const double qmax = (double)code_max(kind, alpha);
    for (uint32_t i = 0; i < n; ++i) {
        double r;
        if (kind == ORC_CODEC_LINEAR) {
            float v = g[i] / scale; /* IEEE fp32 division */
            r = (double)rintf(v);
        } else {
            double mag = rint((double)alpha * log1p(fabs((double)g[i])));
            r = signbit(g[i]) ? -mag : mag;
        }
        if (r > qmax) r = qmax;
        if (r < -qmax) r = -qmax;
        q[i] = (int8_t)r;
    }
    return 0;
}

static float dequant_one(int8_t q, int kind, float scale, float alpha)
{
    if (kind == ORC_CODEC_LINEAR) return (float)((double)q * (double)scale);
    double mag = expm1(fabs((double)q) / (double)alpha);
    return (float)(q < 0 ? -mag : mag);
}

int orc_dequantize(const int8_t* q, float* g, uint32_t n, int kind, float scale, float alpha)
{
    if (!codec_ok(kind, scale, alpha)) return -2;
    const int qmax = code_max(kind, alpha);
    for (uint32_t i = 0; i < n; ++i)
        if (q[i] == -128 || q[i] > qmax || q[i] < -qmax) return -2;
    for (uint32_t i = 0; i < n; ++i) g[i] = dequant_one(q[i], kind, scale, alpha);
    return 0;
}

/* Weight of one perturbation in the apply loop: -grad * eta / numel, where the
 * caller has already folded eta / numel(all_grads) into lr. */
int orc_coefficients(const int8_t* q, uint32_t K, int kind, float scale, float alpha,
                     float lr, float* c)
{
    if (!isfinite(lr)) return -2;
    float* g = c; /* dequantize in place, then scale */
    int rc = orc_dequantize(q, g, K, kind, scale, alpha);
    if (rc) return rc;
    for (uint32_t k = 0; k < K; ++k) c[k] = (float)(-(double)lr * (double)g[k]);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Element-wise operations.                                                 */
/* ------------------------------------------------------------------------ */

static int elems_ok(int dtype, const uint64_t* idx, uint64_t first, uint64_t n)
{
    if (dtype != ORC_F32 && dtype != ORC_BF16) return 0;
    if (idx) {
        for (uint64_t i = 0; i < n; ++i)
            if (idx[i] >> 34) return 0;
    } else if (n > 0 && (first + n - 1) >> 34) {
        return 0;
    }
    return 1;
}

/* PerturbParameters(theta, eps, s): theta_i <- theta_i + eps * z_i. */
int orc_perturb(void* theta, int dtype, uint32_t tensor_id, const uint64_t* idx,
                uint64_t first, uint64_t n, orc_seed_t s, float scale)
{
    if (!elems_ok(dtype, idx, first, n)) return -1;
    if (!isfinite(scale)) return -2;
    if (scale == 0.0f) return 0;
    long long nn = (long long)n;
#pragma omp parallel for schedule(static)
    for (long long i = 0; i < nn; ++i) {
        uint64_t e = idx ? idx[i] : first + (uint64_t)i;
        double v = load_theta(theta, dtype, (uint64_t)i);
        v = v + (double)scale * (double)orc_z(s, tensor_id, e); /* product exact */
        store_theta(theta, dtype, (uint64_t)i, v);
    }
    return 0;
}

/* The apply loop for one iteration: for each (machine, sample) in order,
 * PerturbParameters(theta, -grad*lr, s). The K products c*z are exact in
 * fp64; they are summed in fp64 in ascending k and rounded to storage once. */
int orc_update(void* theta, int dtype, uint32_t tensor_id, const uint64_t* idx,
               uint64_t first, uint64_t n, const orc_seed_t* seeds, const int8_t* q,
               uint32_t K, int kind, float scale, float alpha, float lr)
{
    if (!elems_ok(dtype, idx, first, n)) return -1;
    if (K > 0 && (!seeds || !q)) return -1;
    float* c = (float*)malloc(((size_t)K + 1) * sizeof(float));
    if (!c) return -1;
    int rc = orc_coefficients(q, K, kind, scale, alpha, lr, c);
    uint32_t live = 0;
    for (uint32_t k = 0; rc == 0 && k < K; ++k) live += (c[k] != 0.0f);
    if (rc || live == 0) { /* a zero weight perturbs nothing */
        free(c);
        return rc;
    }
    long long nn = (long long)n;
#pragma omp parallel for schedule(static)
    for (long long i = 0; i < nn; ++i) {
        uint64_t e = idx ? idx[i] : first + (uint64_t)i;
        double acc = 0.0;
        for (uint32_t k = 0; k < K; ++k) {
            if (c[k] == 0.0f) continue;
            acc += (double)c[k] * (double)orc_z(seeds[k], tensor_id, e);
        }
        double v = load_theta(theta, dtype, (uint64_t)i) + acc;
        store_theta(theta, dtype, (uint64_t)i, v);
    }
    free(c);
    return 0;
}

/* Late-joiner catch-up (Appendix B): apply every logged iteration in turn. */
int orc_replay(void* theta, int dtype, uint32_t tensor_id, const uint64_t* idx,
               uint64_t first, uint64_t n, const orc_seed_t* seeds, const int8_t* q,
               const uint32_t* K_t, const float* lr_t, uint32_t T,
               int kind, float scale, float alpha)
{
    uint64_t off = 0;
    for (uint32_t t = 0; t < T; ++t) {
        int rc = orc_update(theta, dtype, tensor_id, idx, first, n, seeds + off, q + off,
                            K_t[t], kind, scale, alpha, lr_t[t]);
        if (rc) return rc;
        off += K_t[t];
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Portable mode: z from binary32 operations only (Appendix B asks for noise */
/* that every device reproduces; hardware transcendentals differ between    */
/* devices, IEEE +, *, fma, / and sqrt do not). The header gives the steps.  */
/* ------------------------------------------------------------------------ */

static void box_muller_pair_portable(uint32_t wa, uint32_t wb, float* zc, float* zs)
{
    /* -2 ln u1 with u1 = n1 2^-24: reduce n1 to m in [sqrt(1/2), sqrt(2)) times
     * a power of two, then ln m = 2 atanh(s), s = (m - 1)/(m + 1). */
    uint32_t n1 = (wa >> 8) + 1u;
    int e = 0;
    while ((n1 >> (e + 1)) != 0u) ++e;                 /* floor(log2 n1) */
    float m = ldexpf((float)n1, -e);                    /* exact, [1, 2) */
    if (m >= 0x1.6a09e6p+0f) {                          /* fl32(sqrt 2) */
        m = m * 0.5f;
        e = e + 1;
    }
    float f = m - 1.0f;                                 /* exact */
    float s = f / (f + 2.0f);
    float s2 = s * s;
    float p = fmaf(s2, 0x1.c71c72p-4f, 0x1.24924ap-3f); /* 1/9, 1/7 */
    p = fmaf(s2, p, 0x1.99999ap-3f);                    /* 1/5 */
    p = fmaf(s2, p, 0x1.555556p-2f);                    /* 1/3 */
    p = fmaf(s2, p, 1.0f);
    float ln_m = (s + s) * p;
    float ln_u1 = fmaf((float)(e - 24), 0x1.62e430p-1f, ln_m); /* + (e-24) ln 2 */
    float r = sqrtf(-2.0f * ln_u1);

    /* (cos, sin)(2 pi u2), u2 = t 2^-24: octant q of v = 8 u2, angle within it */
    uint32_t t = wb >> 8;
    float v = ldexpf((float)t, -21);                    /* exact, [0, 8) */
    int q = (int)v;                                     /* floor, v >= 0 */
    float x = v - (float)q;                             /* exact, [0, 1) */
    float y = (q & 1) ? 1.0f - x : x;                   /* exact, [0, 1] */
    float a = y * 0x1.921fb6p-1f;                       /* fl32(pi/4) */
    float a2 = a * a;
    float sn = fmaf(a2, 0x1.71de3ap-19f, -0x1.a01a02p-13f); /* 1/9!, -1/7! */
    sn = fmaf(a2, sn, 0x1.111112p-7f);                  /* 1/5! */
    sn = fmaf(a2, sn, -0x1.555556p-3f);                 /* -1/3! */
    sn = fmaf(a2, sn, 1.0f);
    sn = a * sn;
    float cs = fmaf(a2, -0x1.27e4fcp-22f, 0x1.a01a02p-16f); /* -1/10!, 1/8! */
    cs = fmaf(a2, cs, -0x1.6c16c2p-10f);                /* -1/6! */
    cs = fmaf(a2, cs, 0x1.555556p-5f);                  /* 1/4! */
    cs = fmaf(a2, cs, -0.5f);                           /* -1/2! */
    cs = fmaf(a2, cs, 1.0f);
    /* the angle is q pi/4 + a (q even) or (q+1) pi/4 - a (q odd) */
    int swap = ((q + 1) >> 1) & 1;                      /* octants 1, 2, 5, 6 */
    int neg_cos = ((q + 2) >> 2) & 1;                   /* octants 2..5 */
    int neg_sin = q >> 2;                               /* octants 4..7 */
    float c0 = swap ? sn : cs;
    float s0 = swap ? cs : sn;
    if (neg_cos) c0 = -c0;
    if (neg_sin) s0 = -s0;
    *zc = r * c0;
    *zs = r * s0;
}

void orc_box_muller_portable(const uint32_t w[4], float z[4])
{
    box_muller_pair_portable(w[0], w[1], &z[0], &z[1]);
    box_muller_pair_portable(w[2], w[3], &z[2], &z[3]);
}

void orc_box_muller_portable_blocks(const uint32_t* w, uint64_t n_blocks, float* z)
{
    long long n = (long long)n_blocks;
#pragma omp parallel for schedule(static)
    for (long long b = 0; b < n; ++b) orc_box_muller_portable(w + 4 * b, z + 4 * b);
}

float orc_z_portable(orc_seed_t s, uint32_t tensor_id, uint64_t e)
{
    uint32_t w[4];
    float z[4];
    orc_block_words(s, tensor_id, e, w);
    orc_box_muller_portable(w, z);
    return z[e & 3u];
}

int orc_generate_portable(orc_seed_t s, uint32_t tensor_id, uint64_t first, uint64_t count,
                          float* z)
{
    if (count > 0 && (first + count - 1) >> 34) return -1;
    long long n = (long long)count;
#pragma omp parallel for schedule(static)
    for (long long i = 0; i < n; ++i) z[i] = orc_z_portable(s, tensor_id, first + (uint64_t)i);
    return 0;
}

static float load_theta_f32(const void* theta, int dtype, uint64_t i)
{
    return (float)load_theta(theta, dtype, i); /* exact for both storage types */
}

int orc_perturb_portable(void* theta, int dtype, uint32_t tensor_id, const uint64_t* idx,
                         uint64_t first, uint64_t n, orc_seed_t s, float scale)
{
    if (!elems_ok(dtype, idx, first, n)) return -1;
    if (!isfinite(scale)) return -2;
    if (scale == 0.0f) return 0;
    long long nn = (long long)n;
#pragma omp parallel for schedule(static)
    for (long long i = 0; i < nn; ++i) {
        uint64_t e = idx ? idx[i] : first + (uint64_t)i;
        float acc = fmaf(scale, orc_z_portable(s, tensor_id, e), 0.0f);
        float v = load_theta_f32(theta, dtype, (uint64_t)i) + acc;
        store_theta(theta, dtype, (uint64_t)i, (double)v);
    }
    return 0;
}

int orc_update_portable(void* theta, int dtype, uint32_t tensor_id, const uint64_t* idx,
                        uint64_t first, uint64_t n, const orc_seed_t* seeds, const int8_t* q,
                        uint32_t K, int kind, float scale, float alpha, float lr)
{
    if (!elems_ok(dtype, idx, first, n)) return -1;
    if (K > 0 && (!seeds || !q)) return -1;
    float* c = (float*)malloc(((size_t)K + 1) * sizeof(float));
    if (!c) return -1;
    int rc = orc_coefficients(q, K, kind, scale, alpha, lr, c);
    uint32_t live = 0;
    for (uint32_t k = 0; rc == 0 && k < K; ++k) live += (c[k] != 0.0f);
    if (rc || live == 0) { /* a zero weight perturbs nothing */
        free(c);
        return rc;
    }
    long long nn = (long long)n;
#pragma omp parallel for schedule(static)
    for (long long i = 0; i < nn; ++i) {
        uint64_t e = idx ? idx[i] : first + (uint64_t)i;
        float acc = 0.0f;
        for (uint32_t k = 0; k < K; ++k) {
            if (c[k] == 0.0f) continue;
            acc = fmaf(c[k], orc_z_portable(seeds[k], tensor_id, e), acc);
        }
        float v = load_theta_f32(theta, dtype, (uint64_t)i) + acc;
        store_theta(theta, dtype, (uint64_t)i, (double)v);
    }
    free(c);
    return 0;
}

int orc_replay_portable(void* theta, int dtype, uint32_t tensor_id, const uint64_t* idx,
                        uint64_t first, uint64_t n, const orc_seed_t* seeds, const int8_t* q,
                        const uint32_t* K_t, const float* lr_t, uint32_t T,
                        int kind, float scale, float alpha)
{
    uint64_t off = 0;
    for (uint32_t t = 0; t < T; ++t) {
        int rc = orc_update_portable(theta, dtype, tensor_id, idx, first, n, seeds + off, q + off,
                                     K_t[t], kind, scale, alpha, lr_t[t]);
        if (rc) return rc;
        off += K_t[t];
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Checksum of theta (Algorithm 1, ChecksumMatch: a hash of the weights      */
/* compared with a random peer). The paper fixes no hash; any function every */
/* replica computes identically serves. A sum of per-chunk mixes is order-    */
/* independent, so it is the same however the tensors are grouped.          */
/* ------------------------------------------------------------------------ */

uint64_t orc_fmix64(uint64_t x)
{
    /* MurmurHash3 (Appleby), 64-bit finalizer */
    x ^= x >> 33;
    x *= 0xFF51AFD7ED558CCDull;
    x ^= x >> 33;
    x *= 0xC4CEB9FE1A85EC53ull;
    x ^= x >> 33;
    return x;
}

uint64_t orc_checksum(const void* data, uint64_t nbytes, uint32_t tensor_id)
{
    const unsigned char* b = (const unsigned char*)data;
    const uint64_t kPos = 0x9E3779B97F4A7C15ull;
    const uint64_t kTensor = 0xD1B54A32D192ED03ull;
    uint64_t n_chunks = (nbytes + 7) / 8;
    uint64_t sum = 0;
    for (uint64_t j = 0; j < n_chunks; ++j) {
        uint64_t c = 0;
        for (int k = 0; k < 8; ++k) {
            uint64_t at = j * 8 + (uint64_t)k;
            if (at < nbytes) c |= (uint64_t)b[at] << (8 * k); /* little-endian */
        }
        sum += orc_fmix64(c ^ (j * kPos) ^ ((uint64_t)tensor_id * kTensor));
    }
    return sum;
}

void orc_set_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

int orc_get_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
