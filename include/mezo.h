/*
 * mezo.h — C ABI of libmezo, the MI355X (gfx950) seeded perturbation engine
 * for shared-randomness SPSA fine-tuning ("Just One Byte (per gradient)",
 * arXiv 2306.10015).
 *
 * The engine regenerates every Gaussian perturbation z from a seed instead of
 * storing it, and applies it to a model's parameters in place:
 *   - mezo_perturb       theta += scale * z(seed)          (Algorithm 1,
 *                        PerturbParameters; called with +eps, -2eps, +eps
 *                        around the two forward passes)
 *   - mezo_update_multi  theta -= lr * sum_k g~_k z(seed_k) (Algorithm 1, the
 *                        apply loop over (timestamp, sample_id) in order)
 *   - mezo_replay        T logged updates one after another (Appendix B,
 *                        late-joiner catch-up)
 *   - quantize_projgrad  projected gradient -> one byte (Section 3)
 *
 * Plain C99: no HIP or torch types. Device pointers are plain pointers into
 * memory of the current HIP device; a stream is a hipStream_t passed as void*
 * (NULL = the null stream).
 *
 * What z is. For seed s = (machine, step, sample), tensor id t and element e
 * of that tensor, the four 32-bit words w0..w3 of
 *     Philox4x32-10(key = (lo32(machine), hi32(machine)),
 *                   counter = (e >> 2, t, sample, step))
 * are turned into four Gaussians by Box-Muller on 24-bit uniforms
 *     u1 = ((w_a >> 8) + 1) * 2^-24,  u2 = (w_b >> 8) * 2^-24,
 *     z = sqrt(-2 ln u1) * (cos 2 pi u2, sin 2 pi u2)
 * with (w0, w1) giving elements 4b, 4b+1 and (w2, w3) giving 4b+2, 4b+3.
 * z therefore depends only on (seed, t, e): not on the launch, the grouping
 * of tensors or the storage type. RNG words are bit-exact with any other
 * implementation of this definition; the Gaussians are computed in fp32 with
 * the GPU's transcendental instructions (absolute error below 1e-6 * max|z|).
 *
 * Arithmetic. theta is loaded into fp32 (bf16 exactly), the perturbations are
 * accumulated in fp32 for k ascending, per Box-Muller pair as
 *     cr = c'_k * rho,  acc_c = fma(cr, cos 2 pi u2, acc_c),
 *                       acc_s = fma(cr, sin 2 pi u2, acc_s),
 * where rho = sqrt(-log2 u1) = z's radius / sqrt(2 ln 2) (the constant factor
 * is taken out of the per-element work) and c'_k = fl32(c_k * sqrt(2 ln 2));
 * then theta' = round(theta + acc) to the storage type, round-to-nearest-even;
 * subnormals are kept.
 *
 * Errors. Every int-returning call returns MEZO_OK (0) or a negative MEZO_E*
 * code; no C++ exception leaves the library. All argument checks run before
 * anything is enqueued, so a failed call leaves the parameters untouched. Device faults surface at the caller's next
 * synchronisation (HIP's convention). mezo_strerror() gives a description;
 * for MEZO_EHIP, mezo_last_error() gives the HIP runtime's message of the last
 * failure on the calling thread.
 *
 * Ownership. Parameter memory belongs to the caller (e.g. PyTorch): the
 * library never allocates or frees it. The library owns a paramset's device
 * tensor table and its seed-staging buffers, released by
 * mezo_paramset_destroy. Host arrays passed to any call are read before the
 * call returns and may be reused at once.
 *
 * Threads and streams. Calls on one paramset may come from several host
 * threads (they serialise on a per-paramset lock). Work is ordered only by the
 * stream it is enqueued on: two calls on different streams that touch the
 * same parameters race unless the caller orders the streams. A paramset
 * tracks the last 16 streams it was used on (destroy waits for their work);
 * a call on a 17th stream first waits on the host for the work of the one
 * used longest ago. mezo_paramset_destroy must not overlap other calls on
 * the same paramset.
 *
 * Graph capture. After a paramset's first call (which creates its device
 * tables), calls that apply at most 32 records, the checksum and the NF4
 * conversions are plain kernel launches and can be captured into a HIP
 * graph; every launch of the graph applies the same records again. The
 * library does not track a graph's launches: synchronize with them before
 * mezo_paramset_destroy. During capture, a paramset's first call and a
 * call with more than 32 records (staged through host memory) fail with
 * MEZO_EINVAL before enqueuing anything.
 */
#ifndef MEZO_H
#define MEZO_H

#include <stdint.h>

#if defined(__GNUC__) || defined(__clang__)
#define MEZO_API __attribute__((visibility("default")))
#else
#define MEZO_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

/* ---- return codes ---------------------------------------------------- */
#define MEZO_OK        0
#define MEZO_EINVAL   -1  /* null/misaligned pointer, empty or oversized tensor,
                             duplicated tensor_id, bad shard offset, bad
                             count, a paramset used on another device, a
                             call that a graph capture cannot record         */
#define MEZO_EDTYPE   -2  /* unknown storage type                            */
#define MEZO_EOVERLAP -3  /* two tensors of a paramset share memory          */
#define MEZO_EORDER   -4  /* seeds of one update not strictly ascending      */
#define MEZO_ERANGE   -5  /* q = -128, NaN gradient, non-finite lr/scale,
                             codec parameters out of range, more than 2^32-1
                             perturbation terms in one call                  */
#define MEZO_EHIP     -6  /* HIP runtime failure (see mezo_last_error)       */
#define MEZO_ENOMEM   -7  /* host memory for the call's records or tables
                             could not be allocated                          */

/* ---- storage types and codecs ---------------------------------------- */
#define MEZO_F32  0u      /* IEEE binary32                                    */
#define MEZO_BF16 1u      /* bfloat16: top 16 bits of a binary32              */
#define MEZO_NF4  2u      /* 4-bit NormalFloat in blocks of 64 elements with an
                             fp32 absmax per block (the 4-bit forward-only
                             variant, Section 3, in QLoRA's format, which the
                             paper cites there); see mezo_tensor_t          */

/* NF4 blocks: elements per absmax value. */
#define MEZO_NF4_BLOCK 64u

#define MEZO_CODEC_LINEAR     0u  /* q = clamp(rne(g / scale), -127, 127);
                                     g~ = fl32(q * scale)                     */
#define MEZO_CODEC_SIGNED_LOG 1u  /* q = sign(g) min(qmax, rne(alpha ln(1+|g|)));
                                     g~ = fl32(sign(q) (exp(|q|/alpha) - 1)).
                                     qmax = 127, or the largest k whose
                                     decoding is a finite fp32 when that is
                                     smaller: alpha = 1/ln 2 (a base-2 log)
                                     puts 127 just inside fp32, the natural
                                     log (alpha = 1) stops at 88. Codes with
                                     |q| > qmax, and an alpha with qmax = 0,
                                     are MEZO_ERANGE.                         */

/* How z is computed (a property of a training run: every machine must use
 * the same one).
 *  FAST:     hardware transcendentals (v_log, v_sqrt, v_sin, v_cos); z within
 *            1e-6 * max|z| of the exact Box-Muller value; the default. On
 *            MEZO_NF4 storage the quantizer may also round differently (a
 *            hardware reciprocal; in one-record calls the block's values
 *            scaled by 1 / absmax): a code can then differ from the rule
 *            stated with mezo_tensor_t only where x lies within about 2^-22
 *            of a midpoint, and the absmax by a few ulp.
 *  PORTABLE: z and the update from IEEE binary32 +, -, *, fma, correctly
 *            rounded / and sqrt only (Appendix B: noise every device
 *            reproduces), so any IEEE machine computes bit-identical z and
 *            weights; about 2.8x the instructions of FAST (2.0x its time).
 *            Per pair of words:
 *            ln u1 from an exact reduction u1 = m 2^e and the series
 *            2 atanh((m-1)/(m+1)), r = sqrt(-2 ln u1), and cos/sin of 2 pi u2
 *            from its octant and Taylor polynomials on [0, pi/4]; every
 *            coefficient and step is fixed in binary32. */
#define MEZO_GAUSS_FAST     0u
#define MEZO_GAUSS_PORTABLE 1u

/* Largest number of elements of one tensor (the counter holds e >> 2 in 32
 * bits). */
#define MEZO_MAX_NUMEL (1ull << 34)

/* A seed (Section 2: built from the machine's identifier/start time, the
 * iteration and the sample index; Algorithm 1 writes it (self_time, t,
 * sample)). A floating-point timestamp is passed as its bit pattern. */
typedef struct {
    uint64_t machine;
    uint32_t step;    /* the iteration t / cur_iter */
    uint32_t sample;  /* index of the projected gradient within its machine's step */
} mezo_seed_t;

/* One parameter tensor: `numel` contiguous elements at device address
 * `data` (16-byte aligned), storage `dtype`. `tensor_id` selects the tensor's
 * noise stream and must be unique within a paramset; keep it stable across
 * machines (e.g. the registration order of the model's parameters).
 *
 * MEZO_NF4: `data` holds ceil(numel / 2) bytes of 4-bit codes, element 2i in
 * the low nibble of byte i (for odd numel the last high nibble is written as
 * 0); `absmax` (16-byte aligned) holds ceil(numel / 64) fp32 values, one per
 * block of 64 consecutive elements (the last block may be shorter). Element e
 * is v[code_e] * absmax[e / 64], v the 16 NF4 values. Every call quantizes
 * again at the end of each step it applies: with w' the block's fp32 values
 * after the step, a' = max |w'|, r = fl32(1 / a') (0 when a' = 0),
 * x = fl32(w' * r), and the new code is the number of NF4 midpoints
 * fl32((v_i + v_{i+1}) / 2) strictly below x (the nearest value, ties to the
 * lower code). For MEZO_F32 and MEZO_BF16 `absmax` must be NULL.
 *
 * `first` is the index, within the logical tensor `tensor_id`, of the element
 * at `data`: 0 for a whole tensor; for a shard of a tensor split across
 * GPUs by element range, the shard's first element. A shard holding elements
 * [first, first + numel) computes exactly the z and the weights of those
 * elements of the whole tensor, and the shards' checksums add up to the whole
 * tensor's. first must be a multiple of 8 with first + numel <=
 * MEZO_MAX_NUMEL; MEZO_NF4 tensors are split by whole tensors only
 * (first = 0). */
typedef struct {
    void*    data;
    uint64_t numel;
    uint32_t tensor_id;
    uint32_t dtype;
    void*    absmax;
    uint64_t first;
} mezo_tensor_t;

/* One-byte gradient code (Section 3). `scale` is used by LINEAR, `alpha` by
 * SIGNED_LOG. */
typedef struct {
    uint32_t kind;
    float    scale;
    float    alpha;
} mezo_codec_t;

/* One logged step of the apply loop (Appendix B): K seeds in ascending
 * (machine, step, sample) order, their one-byte gradients, and the step's
 * per-gradient learning rate (eta_t / numel(all_grads), Algorithm 1). */
typedef struct {
    const mezo_seed_t* seeds;
    const int8_t*      q;
    uint32_t           K;
    float              lr;
} mezo_step_t;

typedef struct mezo_paramset* mezo_paramset_t;

/* ---- parameter sets --------------------------------------------------- */

/* Register n tensors (copied; the array may be reused). Checks: t and out
 * non-null, n >= 1, every data non-null and 16-byte aligned, numel >= 1,
 * first a multiple of 8 (0 for MEZO_NF4) and first + numel <=
 * MEZO_MAX_NUMEL, absmax 16-byte aligned for MEZO_NF4 and NULL otherwise
 * (else MEZO_EINVAL), dtype known (MEZO_EDTYPE), tensor_ids unique
 * (MEZO_EINVAL), no two tensors (codes and absmax arrays included)
 * overlapping in memory (MEZO_EOVERLAP).
 * Device resources are created on the current HIP device at the first launch;
 * every later call must be made with that same device current (MEZO_EINVAL
 * otherwise). */
MEZO_API int mezo_paramset_create(const mezo_tensor_t* t, uint32_t n, mezo_paramset_t* out);

/* Release the paramset's table and staging buffers after waiting for the
 * work it enqueued. NULL is ignored. */
MEZO_API void mezo_paramset_destroy(mezo_paramset_t ps);

/* Total number of elements of a paramset (0 for NULL). */
MEZO_API uint64_t mezo_paramset_numel(mezo_paramset_t ps);

/* Select how z is computed for every later call on ps (MEZO_GAUSS_FAST, the
 * default, or MEZO_GAUSS_PORTABLE; MEZO_EINVAL otherwise). For the *_from
 * calls the destination's setting applies. In portable mode the update is
 *   acc = fma(c_k, z_k, acc) (k ascending, binary32), theta' = round(theta + acc)
 * with the binary32 sum theta + acc rounded to the storage type. A call
 * made while the setting changes on another thread uses one setting
 * throughout, the old or the new. */
MEZO_API int mezo_paramset_set_gaussian(mezo_paramset_t ps, uint32_t gaussian);

/* ---- the engine ------------------------------------------------------- */

/* PerturbParameters(theta, scale, seed) — Algorithm 1: for every element of
 * every tensor, theta <- round(theta + scale * z(seed)). One pass; one read
 * and one write of each element. scale must be finite (MEZO_ERANGE);
 * scale = 0 enqueues nothing. */
MEZO_API int mezo_perturb(mezo_paramset_t ps, mezo_seed_t seed, float scale, void* stream);

/* Several PerturbParameters calls in one pass (Algorithm 1, the loop over
 * samples): for i = 0 .. n-1 in order, theta <- round(theta + scales[i] *
 * z(seeds[i])), rounding to storage after every term — bit-identical to n
 * mezo_perturb calls, for the traffic of one. Between two samples, the restore
 * of sample j (+eps, seed j) and the perturbation for sample j + 1 (+eps,
 * seed j + 1) share one sweep, so a sample costs two sweeps instead of three.
 * Every scale must be finite (MEZO_ERANGE); zero terms are dropped; n = 0 (or
 * nothing left) enqueues nothing; seeds may repeat and need no order. */
MEZO_API int mezo_perturb_multi(mezo_paramset_t ps, const mezo_seed_t* seeds, const float* scales, uint32_t n,
                                void* stream);

/* The apply loop of one iteration — Algorithm 1 and Section 2: in
 * machine/timestamp order, perturb by -grad_k * lr with seed_k. Fused: for
 * every element, acc = sum_k c_k z(seed_k) with c_k = fl32(-lr * g~_k)
 * (g~_k = the codec's decoding of q[k]), then theta <- round(theta + acc);
 * each element is read and written once for all K seeds.
 * seeds must be strictly ascending by (machine, step, sample) (MEZO_EORDER);
 * the fixed order fixes the fp32 sum, so replicas stay bit-identical.
 * q[k] = -128, non-finite lr or a bad codec give MEZO_ERANGE. Terms with
 * c_k = 0 are dropped; K = 0, lr = 0 or all-zero q enqueue nothing. */
MEZO_API int mezo_update_multi(mezo_paramset_t ps, const mezo_seed_t* seeds, const int8_t* q,
                      uint32_t K, const mezo_codec_t* codec, float lr, void* stream);

/* Late-joiner catch-up — Appendix B: apply T logged steps in order, each as
 * mezo_update_multi would (rounding to storage after every step), in one pass
 * over the parameters. Each step is checked as in mezo_update_multi; T = 0
 * enqueues nothing. The result is bit-identical to T mezo_update_multi calls.
 * A log of more than 65536 records runs as several passes, split at step ends
 * (each pass holds at most 65536 records, or one longer step alone); the
 * result is the same, since every step ends rounded to storage anyway. Logs
 * longer than 32 records are staged through host memory in a ring of 4
 * slots: with more passes in flight the call waits on the host for a slot. */
MEZO_API int mezo_replay(mezo_paramset_t ps, const mezo_step_t* steps, uint32_t T,
                const mezo_codec_t* codec, void* stream);

/* mezo_replay for callers that cannot allocate memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation. It makes no
 * device, pinned-host or heap allocation and creates no HIP event: the records
 * (32 B each) go into a file-scope device array of 65536 records (2 MiB) that
 * every GPU the library runs on holds until the process ends, written by small
 * kernels that carry them in their arguments (or, for at most 32 records, into
 * the engine's arguments directly), and the engine reads them from there.
 * Same arguments, checks, arithmetic and result as mezo_replay, bit for bit.
 * Limits and conditions:
 *   - at most 65536 records (non-zero terms) in one call, else MEZO_ERANGE
 *     before anything is enqueued (split a longer log at step ends over
 *     several calls on one stream);
 *   - ps must already have device tables on the current device, which its
 *     first call of any other engine entry point creates (else MEZO_EINVAL);
 *     that set-up also finds the array's address on the device, so this call
 *     makes only kernel launches and may be captured into a HIP graph;
 *   - the array is shared by every call on a GPU and keeps the last call's
 *     records (nothing in it needs clearing: a call writes every record it
 *     reads): two calls whose work may overlap on one GPU — on different
 *     streams without an ordering between them — race; calls on one stream,
 *     or ordered by events, do not. */
MEZO_API int mezo_replay_noalloc(mezo_paramset_t ps, const mezo_step_t* steps, uint32_t T,
                                 const mezo_codec_t* codec, void* stream);

/* Out of place (the weight restore of Algorithm 1 fused into the sweep; it
 * also removes the perturb/restore drift Section 2 mentions): read every
 * tensor of src, write the corresponding tensor of dst, in one pass.
 *   mezo_perturb_from:      theta_dst = round(theta_src + scale * z(seed))
 *   mezo_update_multi_from: theta_dst = round(theta_src + sum_k c_k z(seed_k))
 * src is left unchanged. dst and src must describe the same tensors in the
 * same order (per storage type: numel, tensor_id and first; else MEZO_EINVAL) and
 * share no memory except where a tensor is its own source (MEZO_EOVERLAP);
 * src == dst is the in-place call. Arguments are checked as for the in-place
 * calls. Unlike those, zero weights still enqueue one pass: theta_dst =
 * theta_src (a copy). src's device tables are created on first use, on the
 * same device as dst's. */
MEZO_API int mezo_perturb_from(mezo_paramset_t dst, mezo_paramset_t src, mezo_seed_t seed,
                               float scale, void* stream);
MEZO_API int mezo_update_multi_from(mezo_paramset_t dst, mezo_paramset_t src,
                                    const mezo_seed_t* seeds, const int8_t* q, uint32_t K,
                                    const mezo_codec_t* codec, float lr, void* stream);

/* ---- replica check ----------------------------------------------------- */

/* ChecksumMatch (Algorithm 1): a 64-bit checksum of the bits of every tensor,
 * for comparing replicas (and a late joiner after mezo_replay) with a peer.
 * Each tensor's bytes are read as little-endian 8-byte chunks c_j (the last
 * zero-padded) and
 *   checksum = sum over tensors t, chunks j of
 *              fmix64(c_j ^ j * 0x9E3779B97F4A7C15 ^ tensor_id_t * 0xD1B54A32D192ED03)
 * mod 2^64, fmix64 being MurmurHash3's 64-bit finalizer. The sum does not
 * depend on how tensors are grouped into paramsets or in which order they were
 * registered (the checksum of a model split over several paramsets is the sum
 * of theirs). Chunks are numbered from the start of the logical tensor: a
 * shard (first > 0) starts at chunk first * sizeof(element) / 8, so the
 * checksums of a tensor's shards add up to the whole tensor's. An MEZO_NF4
 * tensor's bytes are its ceil(numel / 2) code bytes
 * zero-padded to a multiple of 8, followed by its absmax values (chunk numbers
 * continue). Written asynchronously to out_dev, a device pointer to 8 bytes
 * (8-byte aligned; MEZO_EINVAL otherwise), on stream. The workgroups sum into
 * a running sum the paramset owns, one per stream it tracks (calls on
 * different streams may overlap), and the call's last workgroup moves the
 * total to out_dev and clears the sum, so no zeroing precedes the call.
 * Calls captured into graphs share one running sum per paramset: replays of
 * such graphs must not overlap in time. */
MEZO_API int mezo_checksum(mezo_paramset_t ps, uint64_t* out_dev, void* stream);

/* ---- 4-bit storage (Section 3, the 4-bit forward-only variant) -------- */

/* Quantize n values of storage src_dtype (MEZO_F32 or MEZO_BF16) at device
 * address src into NF4: ceil(n / 2) code bytes at `codes` and ceil(n / 64)
 * fp32 absmax values at `absmax`, by the rule under mezo_tensor_t. The caller
 * owns all three buffers (device memory, 16-byte aligned, not overlapping;
 * MEZO_EINVAL / MEZO_EDTYPE / MEZO_EOVERLAP otherwise; 1 <= n <=
 * MEZO_MAX_NUMEL). Asynchronous on stream. */
MEZO_API int mezo_nf4_quantize(const void* src, uint32_t src_dtype, uint64_t n, void* codes,
                               float* absmax, void* stream);

/* Dequantize n NF4 elements into dst of storage dst_dtype (MEZO_F32: the
 * value fl32(v[code] * absmax); MEZO_BF16: that value rounded to bf16, to
 * nearest even) — what a forward pass over the 4-bit weights reads. Same
 * ownership, alignment and checks as mezo_nf4_quantize. */
MEZO_API int mezo_nf4_dequantize(const void* codes, const float* absmax, uint64_t n, void* dst,
                                 uint32_t dst_dtype, void* stream);

/* ---- the one-byte gradient (host, pure) ------------------------------- */

/* Projected gradient g = (l+ - l-) / (2 eps) -> q (Section 3). ±inf clip to
 * ±127; NaN is MEZO_ERANGE. Rounding ties go to even. n may be 0. */
MEZO_API int quantize_projgrad(const float* g, int8_t* q, uint32_t n, const mezo_codec_t* codec);

/* q -> g~ (the value every machine applies). q = -128 is MEZO_ERANGE. */
MEZO_API int mezo_dequantize(const int8_t* q, float* g, uint32_t n, const mezo_codec_t* codec);

/* ---- inspection -------------------------------------------------------- */

/* Write the RNG word (words_dev[i] = word e & 3 of the block of element e)
 * and/or the Gaussian z_dev[i] (computed as `gaussian` says) of elements
 * e = first_elem + i, i < count, of tensor tensor_id under seed. Either device
 * pointer may be NULL; first_elem + count <= MEZO_MAX_NUMEL and a known
 * `gaussian` (MEZO_EINVAL). */
MEZO_API int mezo_debug_generate(mezo_seed_t seed, uint32_t tensor_id, uint64_t first_elem,
                                 uint64_t count, uint32_t gaussian, uint32_t* words_dev,
                                 float* z_dev, void* stream);

/* The Gaussian transform alone, on given words: z_dev[4b .. 4b+3] from
 * words_dev[4b .. 4b+3] for b < n_blocks, computed as `gaussian` says — the
 * pair transform above, so that it can be checked over chosen inputs (every
 * value of u1, every value of u2). Both device arrays 16-byte aligned,
 * n_blocks <= 2^32, a known `gaussian` (MEZO_EINVAL otherwise). */
MEZO_API int mezo_debug_box_muller(const uint32_t* words_dev, uint64_t n_blocks, uint32_t gaussian,
                                   float* z_dev, void* stream);

MEZO_API const char* mezo_strerror(int code);

/* The message of the last MEZO_EHIP failure on this thread (the HIP
 * runtime's), or of the last MEZO_ENOMEM or device-mismatch failure ("" if
 * none). */
MEZO_API const char* mezo_last_error(void);

/* Library version, major*10000 + minor*100 + patch. */
MEZO_API int mezo_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MEZO_H */
