/*
 * mezo_oracle.h — CPU oracle for the seeded perturbation engine.
 *
 * TEST INFRASTRUCTURE ONLY. This is a plain, slow, obviously-correct C99
 * statement of what the engine computes. Only the tests, the smoke check and
 * the benchmark's CPU-baseline leg may load or call it; the product path
 * (the HIP library and its Python binding) never does. It shares no code,
 * header, table or constant with the HIP path.
 *
 * What it follows (paper: "Just One Byte (per gradient)", arXiv 2306.10015):
 *  - PerturbParameters (Appendix A, Algorithm 1, the PerturbParameters
 *    subroutine): reset an RNG with seed s, draw z ~ N(0,1) per parameter and
 *    add eps*z to it.
 *  - the perturb / evaluate triple +eps, -2eps, +eps (Algorithm 1, inner
 *    inference loop);
 *  - the apply loop (Algorithm 1, after GetGradients; Section 2): ordered by
 *    machine timestamp, perturb with weight -grad * eta / numel(all_grads)
 *    and the same seed;
 *  - the one-byte gradient (Section 3: a signed log, clipped to +-127);
 *  - late-joiner catch-up (Appendix B): apply every logged projected gradient
 *    of the missed iterations.
 *
 * Readings where the paper is silent:
 *  - the RNG is Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11), keyed by
 *    the machine id, with counter (element>>2, tensor_id, sample, step);
 *  - a Gaussian is Box-Muller on exact 24-bit uniforms, evaluated in fp64 and
 *    rounded once to fp32 (the fp32 sample z_ref);
 *  - perturb/update add in fp64 and round once, straight to the storage type,
 *    round-to-nearest-even; no flush of subnormals anywhere.
 *
 * Parity status: every function here is pinned by the CPU tests (published
 * Philox engine cross-check, closed-form transform cases, statistics,
 * exhaustive codec round trips, brute-force rounding, and the invariants of
 * the update); none is "parity unpinned".
 */
#ifndef MEZO_ORACLE_H
#define MEZO_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* A seed s = (machine start time / id, iteration, sample index), Section 2 and
 * Algorithm 1. Layout: 16 bytes, machine first. */
typedef struct {
    uint64_t machine;
    uint32_t step;
    uint32_t sample;
} orc_seed_t;

enum { ORC_F32 = 0, ORC_BF16 = 1 };
enum { ORC_CODEC_LINEAR = 0, ORC_CODEC_SIGNED_LOG = 1 };

/* Return codes: 0 ok, -1 bad argument, -2 value out of range. */

/* Philox4x32-10 block function: 128-bit counter, 64-bit key -> 4 words. */
void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);

/* The four RNG words of the block that holds element e of tensor tensor_id. */
void orc_block_words(orc_seed_t s, uint32_t tensor_id, uint64_t e, uint32_t out[4]);

/* Box-Muller on one block of four words, fp64: z[0..3] (not rounded). */
void orc_box_muller(const uint32_t w[4], double z[4]);
/* orc_box_muller over n blocks of given words, each z rounded once to fp32. */
void orc_box_muller_blocks(const uint32_t* w, uint64_t n_blocks, float* z);

/* The fp32 Gaussian of element e: fl32 of the fp64 Box-Muller value. */
float orc_z(orc_seed_t s, uint32_t tensor_id, uint64_t e);

/* z_ref and the element's own RNG word for count elements from first. Either
 * output may be NULL. */
int orc_generate(orc_seed_t s, uint32_t tensor_id, uint64_t first, uint64_t count,
                 uint32_t* words, float* z);

/* Direct round-to-nearest-even of an fp64 value to fp32 / bf16 bits. */
float    orc_round_f32(double x);
uint16_t orc_round_bf16(double x);

/* One-byte codec. LINEAR: q = clamp(rne(g/scale), -127, 127),
 *             g~ = fl32(q*scale).
 * SIGNED_LOG: q = sign(g)*min(qmax, rne(alpha*ln(1+|g|))),
 *             g~ = fl32(sign(q)*(exp(|q|/alpha)-1)); alpha = 1/ln 2 is a
 *             base-2 log, alpha = 1 the natural one. qmax is 127, or the
 *             largest k whose decoding fl32(exp(k/alpha) - 1) is finite
 *             when that is smaller (alpha = 1: 88).
 * Rejected with -2: NaN g, q = -128 or |q| > qmax, a non-positive or
 * non-finite scale or alpha, an alpha with qmax = 0. */
int orc_signed_log_qmax(float alpha);
int orc_quantize(const float* g, int8_t* q, uint32_t n, int kind, float scale, float alpha);
int orc_dequantize(const int8_t* q, float* g, uint32_t n, int kind, float scale, float alpha);

/* c_k = fl32(-lr * g~_k): the weight of perturbation k in the apply loop. */
int orc_coefficients(const int8_t* q, uint32_t K, int kind, float scale, float alpha,
                     float lr, float* c);

/*
 * The element-wise operations act on n elements of one tensor. Element i of the
 * buffer `theta` (dtype ORC_F32: float, ORC_BF16: uint16 bits) is tensor
 * element idx[i], or first+i when idx is NULL. Elements must be < 2^34.
 */

/* theta_i <- round_st(theta_i + scale * z_ref_i(s)). scale = 0 is a no-op. */
int orc_perturb(void* theta, int dtype, uint32_t tensor_id, const uint64_t* idx,
                uint64_t first, uint64_t n, orc_seed_t s, float scale);

/* theta_i <- round_st(theta_i + sum_k c_k * z_ref_i(s_k)), sum in fp64 over
 * ascending k, terms with c_k = 0 left out; c_k from orc_coefficients. */
int orc_update(void* theta, int dtype, uint32_t tensor_id, const uint64_t* idx,
               uint64_t first, uint64_t n, const orc_seed_t* seeds, const int8_t* q,
               uint32_t K, int kind, float scale, float alpha, float lr);

/* T logged steps, each an orc_update with its own seeds, q (K_t of each, packed
 * one step after another) and lr_t; storage rounding after every step. */
int orc_replay(void* theta, int dtype, uint32_t tensor_id, const uint64_t* idx,
               uint64_t first, uint64_t n, const orc_seed_t* seeds, const int8_t* q,
               const uint32_t* K_t, const float* lr_t, uint32_t T,
               int kind, float scale, float alpha);

/*
 * Portable mode (Appendix B: the noise must be reproducible on any device).
 * z is defined by a fixed sequence of IEEE binary32 operations (+, -, *, fma,
 * correctly rounded / and sqrt, exact scalings; round-to-nearest-even), so
 * every IEEE machine computes it bit for bit:
 *   n1 = (w_a >> 8) + 1, e = floor(log2 n1), m = n1 * 2^-e in [1, 2);
 *   if m >= fl32(sqrt 2): m = m/2, e = e+1;
 *   f = m - 1; s = f / (f + 2); s2 = s*s;
 *   p = fma(s2, fma(s2, fma(s2, fma(s2, 1/9, 1/7), 1/5), 1/3), 1);
 *   ln_u1 = fma(e - 24, fl32(ln 2), (s + s) * p);     [ln m = 2 atanh s]
 *   r = sqrt(-2 * ln_u1);
 *   v = (w_b >> 8) * 2^-21 (= 8 u2); q = floor v; x = v - q;
 *   y = q odd ? 1 - x : x; a = y * fl32(pi/4); a2 = a*a;
 *   sin a = a * (1 + a2(-1/3! + a2(1/5! + a2(-1/7! + a2/9!))))   (Horner, fma),
 *   cos a = 1 + a2(-1/2! + a2(1/4! + a2(-1/6! + a2(1/8! - a2/10!))));
 *   octant q maps (cos a, sin a) to (cos 2 pi u2, sin 2 pi u2) by swaps
 *   and sign flips; z = (r cos, r sin).
 * (all coefficients rounded to binary32). The update then accumulates in
 * binary32 as acc = fma(c_k, z_k, acc) for k ascending (zero c_k skipped) and
 * theta' = round_st(theta + acc) with the sum in binary32.
 */
void  orc_box_muller_portable(const uint32_t w[4], float z[4]);
/* orc_box_muller_portable over n blocks of given words. */
void  orc_box_muller_portable_blocks(const uint32_t* w, uint64_t n_blocks, float* z);
float orc_z_portable(orc_seed_t s, uint32_t tensor_id, uint64_t e);
int   orc_generate_portable(orc_seed_t s, uint32_t tensor_id, uint64_t first, uint64_t count,
                            float* z);
int   orc_perturb_portable(void* theta, int dtype, uint32_t tensor_id, const uint64_t* idx,
                           uint64_t first, uint64_t n, orc_seed_t s, float scale);
int   orc_update_portable(void* theta, int dtype, uint32_t tensor_id, const uint64_t* idx,
                          uint64_t first, uint64_t n, const orc_seed_t* seeds, const int8_t* q,
                          uint32_t K, int kind, float scale, float alpha, float lr);
int   orc_replay_portable(void* theta, int dtype, uint32_t tensor_id, const uint64_t* idx,
                          uint64_t first, uint64_t n, const orc_seed_t* seeds, const int8_t* q,
                          const uint32_t* K_t, const float* lr_t, uint32_t T,
                          int kind, float scale, float alpha);

/* Checksum of a tensor's bits (ChecksumMatch, Algorithm 1: replicas compare a
 * hash of theta). The tensor's nbytes bytes are read as little-endian 8-byte
 * chunks c_j, the last one zero-padded; the result is
 *     sum_j fmix64(c_j ^ (j * P1) ^ (tensor_id * P2))  mod 2^64
 * with P1 = 0x9E3779B97F4A7C15, P2 = 0xD1B54A32D192ED03 and fmix64 the 64-bit
 * finalizer of MurmurHash3. A parameter set's checksum is the sum over its
 * tensors, so it does not depend on grouping or order. */
uint64_t orc_fmix64(uint64_t x);
uint64_t orc_checksum(const void* data, uint64_t nbytes, uint32_t tensor_id);

/* Thread control for the OpenMP loops (1 when built without OpenMP). */
void orc_set_threads(int n);
int  orc_get_threads(void);

#ifdef __cplusplus
}
#endif

#endif /* MEZO_ORACLE_H */
