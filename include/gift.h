/*
 * gift.h -- C ABI of the GIFT gradient codec for AMD Instinct MI355X (gfx950).
 *
 * GIFT ("Geometry-Informed Low-precision Gradient Communication") communicates
 * each weight gradient W_g in R^{d_out x d_in} (Sec. IV-A, eq. design_Wg) in FP8
 * after mapping it into near-isotropic coordinates built from K-FAC factors
 * (Sec. II-B, eq. kfac_fisher_block; Sec. IV-A, eq. design_full_transform and
 * design_input_side_transform), then maps the synchronized result back
 * (eq. design_full_inverse_transform / design_input_side_inverse).  This
 * library is the per-layer hot path of that rule (Algorithm 1) on one GPU:
 *
 *   gift_factor_update   factor statistics A = E[a a^T], G = E[delta delta^T]
 *                        and their rank-r transforms (Sec. V-B, eq. impl_A_lowrank)
 *   gift_encode          transform, amax scale, FP8 E4M3 quantize (Algorithm 1)
 *   gift_reduce_local    dequantize and average the N data-parallel ranks held
 *                        on this GPU (eq. dp_grad_avg; Algorithm 1 sum and /N)
 *   gift_decode          inverse transform of the averaged gradient
 *
 * Notation: m = d_out (rows), n = d_in (columns), N data-parallel ranks, r the
 * transform rank, T tokens behind the factor statistics.
 *
 * Conventions shared by every call
 * --------------------------------
 * - Tensors are DEVICE pointers, row-major and densely packed, allocated and
 *   owned by the caller.  The library owns only the opaque gift_ctx and
 *   gift_factor objects and the device workspace inside them.
 * - Every compute call validates its arguments on the host, then enqueues
 *   kernels on the context's HIP stream and returns without synchronizing.
 *   A non-GIFT_OK status means nothing was enqueued, except GIFT_EHIP, which
 *   reports a HIP runtime error seen while enqueueing.
 * - gift_last_error() returns a thread-local message describing the last
 *   non-OK status of the calling thread.  No C++ exception crosses the ABI.
 * - Calls on one context are not thread-safe; use one context per host thread.
 * - Block scaling: each rank's m x n matrix is tiled into blocks of
 *   block_rows x block_cols elements (0 = the whole dimension; partial edge
 *   blocks allowed), nbr = ceil(m / block_rows), nbc = ceil(n / block_cols).
 *   Scales are stored as float32 [N, nbr, nbc].
 * - FP8 codes are OCP E4M3 (E4M3FN) bit patterns: bias 7, largest finite 448,
 *   NaN = 0x7F/0xFF, no infinities.  Quantization is
 *       s   = fl32(amax / 448)           (stored scale)
 *       y   = fl32(x * fl32(448 / amax)) (amax = 0 -> multiplier 0; an
 *                                         overflowing multiplier -> FLT_MAX)
 *       q   = round-to-nearest-even E4M3(y), saturating at +-448, keeping the
 *             sign of zero, NaN -> 0x7F.
 *   amax is the exact block maximum of |x|; a NaN in a block makes its amax
 *   (and scale) NaN.
 */
#ifndef GIFT_H
#define GIFT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GIFT_ABI_VERSION 1

typedef struct gift_ctx gift_ctx;
typedef struct gift_factor gift_factor;

typedef enum {
  GIFT_OK = 0,
  GIFT_EINVAL = -1,        /* NULL handle/pointer, bad enum, bad count        */
  GIFT_ESHAPE = -2,        /* sizes inconsistent or out of the supported range */
  GIFT_ENOMEM = -3,        /* device or host allocation failed                */
  GIFT_EHIP = -4,          /* HIP runtime error while enqueueing              */
  GIFT_EUNSUPPORTED = -5   /* valid request the library does not implement   */
} gift_status;

typedef enum { GIFT_F32 = 0, GIFT_BF16 = 1 } gift_dtype;

/* Which sides of the K-FAC geometry a factor applies (Sec. IV-A, V-A). */
enum {
  GIFT_SIDE_INPUT = 1,   /* right factor from A (d_in x d_in): W S_A^-1      */
  GIFT_SIDE_OUTPUT = 2,  /* left factor from G (d_out x d_out): S_G^-1 W     */
  GIFT_SIDE_BOTH = 3     /* both: S_G^-1 W S_A^-1                             */
};

/* Scale mode (Algorithm 1): LOCAL keeps each rank's own amax (the GIFT
 * branch's local scaling, Sec. V-E); SHARED takes the maximum over the N ranks
 * first (the AllReduce_MAX of the Euclidean branch and of scale-sync steps). */
typedef enum { GIFT_SCALE_LOCAL = 0, GIFT_SCALE_SHARED = 1 } gift_scale_mode;

/* Kernel families, for the optional per-kernel timing below. */
typedef enum {
  GIFT_KERNEL_AMAX = 0,          /* Euclidean block amax                     */
  GIFT_KERNEL_QUANT = 1,         /* Euclidean scale + FP8 pack               */
  GIFT_KERNEL_PROJECT = 2,       /* W U_A and U_G^T W projections             */
  GIFT_KERNEL_UPDATE_AMAX = 3,   /* rank-r update fused with block amax       */
  GIFT_KERNEL_UPDATE_QUANT = 4,  /* rank-r update fused with scale + FP8 pack */
  GIFT_KERNEL_UPDATE_STORE = 5,  /* rank-r update of the inverse transform    */
  GIFT_KERNEL_REDUCE = 6,        /* dequantize-accumulate over ranks          */
  GIFT_KERNEL_SYRK = 7,          /* factor statistics X^T X / T               */
  GIFT_KERNEL_FACTOR = 8,        /* subspace-iteration products and setup     */
  GIFT_KERNEL_SMALL = 9,         /* small helpers (zeroing, coefficient setup) */
  GIFT_KERNEL_CHOL = 10,         /* CholeskyQR's k x k Cholesky and R^-1      */
  GIFT_KERNEL_EIG = 11,          /* Rayleigh-Ritz k x k eigensolver           */
  GIFT_KERNEL_DECODE_PROJECT = 12, /* the inverse transform's projections     */
  GIFT_KERNEL_CHOL_TRANSFORM = 13, /* Cholesky-form transform products         */
  GIFT_KERNEL_MXFP4 = 14,        /* MXFP4 scale + pack (gift_encode_mxfp4)     */
  GIFT_KERNEL_COUNT = 15
} gift_kernel;

/* ABI version of the loaded library (GIFT_ABI_VERSION it was built with). */
int32_t gift_abi_version(void);

/* Thread-local description of the calling thread's last non-OK status. */
const char *gift_last_error(void);

/* Create a context bound to a HIP stream (hipStream_t passed as void*; NULL is
 * the null stream).  No HIP call is made until the first compute call, which
 * binds the context to the then-current device.  *out receives the handle. */
gift_status gift_ctx_create(void *hip_stream, gift_ctx **out);

/* Rebind the context to another stream of the same device.  Work already
 * queued on the old stream is waited for first: the context's scratch memory
 * is ordered by the stream it was used on. */
gift_status gift_ctx_set_stream(gift_ctx *ctx, void *hip_stream);

/* Destroy a context (synchronizes its stream, frees its workspace). NULL ok.
 * Destroy the factors created on it first. */
void gift_ctx_destroy(gift_ctx *ctx);

/* Scheduling hook: every later gift_factor_update[_batch] call on this
 * context records hip_event (a hipEvent_t passed as void*, created and owned
 * by the caller) on the context stream right after its statistics kernels
 * (A = X^T X / T of every factor side), before the rest of the refresh.
 * Other streams can wait on it to start work once the statistics (the
 * refresh's compute-bound part) are done.  NULL stops the recording.  The
 * event must stay valid until it is replaced or unset (the library keeps the
 * handle, not a copy).  For the Cholesky-form factors nothing is recorded.
 * Errors: GIFT_EINVAL for a NULL ctx. */
gift_status gift_ctx_set_statistics_event(gift_ctx *ctx, void *hip_event);

/* Per-kernel timing: when enabled, every launch of a selected kernel family
 * is bracketed by HIP events on the context stream (all families are selected
 * until gift_ctx_profile_select is called).  gift_ctx_profile_read
 * synchronizes the stream and returns the number of launches and their summed
 * duration (ms) for one kernel family since the last reset;
 * gift_ctx_profile_reset clears the counters.  family_mask: bit k selects
 * kernel family k (gift_kernel). */
gift_status gift_ctx_profile_enable(gift_ctx *ctx, int32_t enable);
gift_status gift_ctx_profile_select(gift_ctx *ctx, uint32_t family_mask);
gift_status gift_ctx_profile_read(gift_ctx *ctx, int32_t kernel, int64_t *launches,
                                  double *total_ms);
gift_status gift_ctx_profile_reset(gift_ctx *ctx);

/* Create the transform state of one m x n weight matrix (Algorithm 1's
 * per-layer factor).  rank: r >= 0 (r <= n for the input side, r <= m for the
 * output side; 0 = identity).  sides: GIFT_SIDE_*.  damping: relative floor of
 * the isotropic level sigma^2 (>= damping * tr(A)/n), the regularization of
 * eq. design_chol.  seed: key of the Philox4x32-10 start block of the subspace
 * iteration (input side: seed; output side: seed + 1).  The new factor is the
 * identity until updated or imported.
 * Allocates device memory on the current device (synchronous). */
gift_status gift_factor_create(gift_ctx *ctx, int64_t m, int64_t n, int32_t rank,
                               int32_t sides, float damping, uint64_t seed,
                               gift_factor **out);

/* Create a Cholesky-form factor (Sec. IV-A, eq. design_chol with the
 * transforms of eq. design_full_transform / design_input_side_transform and
 * their inverses; Table II's full-A, diag-A and block-A-b variants):
 *   A + delta I = L_A L_A^T,  delta = damping * tr(A) / n  (G likewise, dim m),
 *   encode W~ = L_G^-1 W L_A^-T,  decode W^ = L_G M L_A^T.
 * block: 0 (or >= dim) = the full Cholesky factor; 1 = the diagonal of A
 * (L = diag(sqrt(a_ii + delta))); b >= 2 = the Cholesky factors of the b x b
 * diagonal blocks of A + delta I (the last block ragged when b does not
 * divide dim), L block-diagonal.  A side's effective block is
 * b_eff = min(block or dim, dim); it is stored as nblk = ceil(dim / b_eff)
 * blocks of b_eff x b_eff (gift_factor_export_chol).
 * damping must be > 0 (every pivot is then at least delta); a zero trace
 * gives the identity.  gift_factor_update refreshes it from the statistics
 * (iters is ignored); gift_encode, gift_encode_hits and gift_decode apply it
 * (float32 products; the FP8 step is the Euclidean encode of W~).  The new
 * factor is the identity.  Blocks above 128 are factored by one workgroup
 * each: the full factor of a large dim is a slow refresh.
 * Errors: GIFT_EINVAL (NULL, bad sides, damping not finite and > 0),
 * GIFT_ESHAPE (m, n out of range, block < 0, block_eff > 8192). */
gift_status gift_factor_create_chol(gift_ctx *ctx, int64_t m, int64_t n, int32_t block,
                                    int32_t sides, float damping, gift_factor **out);

/* Destroy a factor (synchronizes the context stream first). NULL ok.  A
 * factor must be destroyed before the context it was created on. */
void gift_factor_destroy(gift_factor *f);

/* Refresh the factor from one batch of statistics (Sec. V-E: refreshed every
 * K steps; Algorithm 1's A ~ L_A L_A^T).
 *   acts       [T, n] layer inputs a (device; float32 or bfloat16 per dtype),
 *              required when sides include GIFT_SIDE_INPUT, else ignored;
 *   out_grads  [T, m] gradients delta w.r.t. the layer outputs, required when
 *              sides include GIFT_SIDE_OUTPUT, else ignored;
 *   iters      subspace iterations (>= 0).  The first update starts from the
 *              Philox block; later updates warm-start from the previous
 *              subspace.
 * Computes A = acts^T acts / T (and G likewise), its top-r eigenpairs by
 * block subspace iteration (k = min(dim, 2r) columns, CholeskyQR2) with
 * Rayleigh-Ritz extraction, sigma^2 = mean of the remaining eigenvalues
 * (floored at damping * tr/dim), and the coefficients
 *   c_i = sqrt(sigma^2/lambda_i) - 1,  c'_i = sqrt(lambda_i/sigma^2) - 1,
 * so that S^-1 = I + U diag(c) U^T and S = I + U diag(c') U^T. */
gift_status gift_factor_update(gift_ctx *ctx, gift_factor *f, const void *acts,
                               const void *out_grads, int64_t T, gift_dtype dtype,
                               int32_t iters);

/* Factor statistics alone (eq. kfac_fisher_block, eq. impl_A_psd): the
 * uncentred second moment A = X^T X / T of one statistics input, the first
 * step of gift_factor_update.
 *   x  [T, dim] row-major, float32 or bfloat16 per dtype (device);
 *   A  [dim, dim] float32 out (device), full symmetric matrix.
 * bfloat16 products are exact in float32 and every sum is accumulated in
 * float32.  Uses the context workspace. */
gift_status gift_statistics(gift_ctx *ctx, const void *x, int64_t T, int64_t dim, gift_dtype dtype,
                            float *A);

/* Refresh many factors at once (same T and dtype): factor sides with equal
 * (dim, rank) share one launch sequence, so the small per-factor steps run
 * side by side on the GPU.  factors, acts and out_grads are HOST arrays of
 * count entries; acts[i] / out_grads[i] are the device inputs of factors[i]
 * (an entry may be NULL when that factor lacks the side; the whole array may
 * be NULL when no factor has the side).  A factor may appear only once.
 * Results equal count separate gift_factor_update calls. */
gift_status gift_factor_update_batch(gift_ctx *ctx, int32_t count, gift_factor *const *factors,
                                     const void *const *acts, const void *const *out_grads,
                                     int64_t T, gift_dtype dtype, int32_t iters);

/* Copy one side's transform out of / into a factor (device pointers):
 *   U [dim, r] row-major (dim = n for GIFT_SIDE_INPUT, m for GIFT_SIDE_OUTPUT),
 *   c_fwd [r], c_inv [r], sigma2 [1].
 * side must be GIFT_SIDE_INPUT or GIFT_SIDE_OUTPUT and present in the factor.
 * Import replaces the side's transform (the next update warm-starts from
 * U).  Enqueued on the context stream.  GIFT_EINVAL for a Cholesky-form
 * factor (gift_factor_export_chol / gift_factor_import_chol). */
gift_status gift_factor_export(gift_ctx *ctx, const gift_factor *f, int32_t side,
                               float *U, float *c_fwd, float *c_inv, float *sigma2);
gift_status gift_factor_import(gift_ctx *ctx, gift_factor *f, int32_t side,
                               const float *U, const float *c_fwd, const float *c_inv,
                               const float *sigma2);

/* Encode the N ranks' gradients (Algorithm 1, both branches):
 *   f            factor of this m x n matrix, or NULL for the Euclidean branch;
 *   grads        [N, m, n] float32 rank gradients;
 *   mode         GIFT_SCALE_LOCAL or GIFT_SCALE_SHARED;
 *   ef           error-feedback residual [N, m, n] float32 in transformed
 *                coordinates (Algorithm 1: U~ = U + R; R <- U~ - Deq(Q(U~))),
 *                or NULL for none.  Zero it before the first step;
 *   codes        [N, m, n] uint8 out: E4M3 codes of W~_j = S_G^-1 W_j S_A^-1 (+R)
 *                (L_G^-1 W_j L_A^-T for a Cholesky-form factor);
 *   scales       [N, nbr, nbc] float32 out;
 *   transformed  optional [N, m, n] float32 out: W~ (+R) before quantization.
 * Output buffers must not overlap the inputs. */
gift_status gift_encode(gift_ctx *ctx, const gift_factor *f, const float *grads,
                        int32_t N, int64_t m, int64_t n, int32_t block_rows,
                        int32_t block_cols, gift_scale_mode mode, float *ef,
                        uint8_t *codes, float *scales, float *transformed);

/* Size of the fixed device scratch of gift_encode_noalloc (64 MiB per device). */
#define GIFT_NOALLOC_SCRATCH_BYTES (64ull * 1024ull * 1024ull)

/* gift_encode without any device allocation, for callers that cannot
 * allocate: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  Arguments, results and kernels are those of gift_encode
 * (codes, scales, ef and transformed identical).  Its scratch (block-maximum
 * sub-slots, the finalize buffer, the projections P = W U and their partial
 * sums, a stored W~ when the transform cannot be recomputed, the Cholesky-form
 * transform buffer) comes from one fixed array of GIFT_NOALLOC_SCRATCH_BYTES
 * in device memory, which each device holds from the library's load there
 * until the process ends; the call makes no hipMalloc, hipFree, event or
 * other allocating call (the first call on a device looks the array's device
 * address up once).  The sub-slots are cleared by a kernel at the start of
 * every call.  Limits: a call whose scratch exceeds the array returns
 * GIFT_ESHAPE before anything is enqueued (e.g. a low-rank encode needs about
 * 4 N m r (parts + 1) bytes of projections; split the ranks or rows, or pass
 * `transformed` where W~ would be stored).  Every call on one device shares
 * the array: calls that overlap in time on one device (other streams, other
 * contexts, other threads) race and must be ordered by the caller.  The
 * context's device must be current.  Per-kernel timing is not recorded. */
gift_status gift_encode_noalloc(gift_ctx *ctx, const gift_factor *f, const float *grads,
                                int32_t N, int64_t m, int64_t n, int32_t block_rows,
                                int32_t block_cols, gift_scale_mode mode, float *ef,
                                uint8_t *codes, float *scales, float *transformed);

/* Copy one side of a Cholesky-form factor out of / into it (device
 * pointers): R and Rinv are [nblk, b_eff, b_eff] float32, block k holding
 * R_k = L_k^T (upper triangular) and its inverse; the last block's kv x kv
 * part (kv = dim - (nblk - 1) b_eff) sits top-left, the identity elsewhere.
 * Import replaces the side (both arrays are read as given).  Errors:
 * GIFT_EINVAL for a low-rank factor, a side the factor lacks or NULL arrays. */
gift_status gift_factor_export_chol(gift_ctx *ctx, const gift_factor *f, int32_t side, float *R,
                                    float *Rinv);
gift_status gift_factor_import_chol(gift_ctx *ctx, gift_factor *f, int32_t side, const float *R,
                                    const float *Rinv);

/* gift_encode plus per-rank counters of codes that sit at either end of the
 * FP8 range (Sec. V-C: the per-layer numerical-vulnerability profile
 * that selects the layers for the geometry-aware branch; the score is the sum
 * of the two ratios, i.e. of a rank's two counts over m*n):
 *   hits[2j]   += codes of rank j with magnitude 448, the largest finite E4M3
 *                 value (saturated values and every block's maximum itself);
 *   hits[2j+1] += nonzero values of rank j whose code is +-0 (after scaling
 *                 at most half the smallest subnormal, 2^-10).
 * The counted values are those the codes encode (W~, + R with error
 * feedback); NaN values count in neither.  hits: device, 4-byte aligned,
 * uint32 [N][2], accumulated across calls (the caller zeroes it); counts past
 * 2^32 - 1 wrap.  Everything else as gift_encode; the counting is done by the
 * quantize kernels as they pack (no extra pass over the tensors).
 * Errors: as gift_encode; GIFT_EINVAL for a NULL or misaligned hits. */
gift_status gift_encode_hits(gift_ctx *ctx, const gift_factor *f, const float *grads,
                             int32_t N, int64_t m, int64_t n, int32_t block_rows,
                             int32_t block_cols, gift_scale_mode mode, float *ef,
                             uint8_t *codes, float *scales, float *transformed,
                             uint32_t *hits);

/* MXFP4 variant of gift_encode: the same transform (W~ = S_G^-1 W S_A^-1, or
 * the Cholesky form; f = NULL: W itself), then OCP Microscaling FP4 instead of
 * FP8 -- the 4-bit format the paper names as future work (Sec. I; Sec. VI,
 * Discussion):
 *   per rank, row and 32 consecutive columns, k = floor(log2(amax)) - 2
 *   (>= -127; a block holding a NaN or an infinity: scale 255 = NaN, codes 0),
 *   scales = k + 127 (E8M0), each element v * 2^-k rounded to the nearest FP4
 *   E2M1 value (0, 0.5, 1, 1.5, 2, 3, 4, 6; ties to the even code; larger
 *   magnitudes saturate to 6; sign of zero kept).
 *   codes  [N, m, n/2] uint8 out, two codes per byte, element 2i in the low
 *          nibble (4-byte aligned);  scales [N, m, n/32] uint8 out;
 *   ef     optional residual [N, m, n] in transformed coordinates, read and
 *          rewritten (U = W~ + R; R <- U - Dequantize(codes));
 *   transformed  optional [N, m, n] float32 out: U before quantization.
 * The low-rank transform is computed as in gift_encode (split-bf16 products)
 * and packed in the same pass when the rank is a multiple of 4 and at most
 * 128 and one rank's slice has fewer than 2^29 elements; otherwise W~ is
 * stored with float32 products, then quantized.  n must be a multiple of 32 (GIFT_ESHAPE); grads, ef and
 * transformed 16-byte aligned (GIFT_EINVAL).  Scales are per rank (no
 * shared-scale mode).  Uses the context workspace. */
gift_status gift_encode_mxfp4(gift_ctx *ctx, const gift_factor *f, const float *grads, int32_t N,
                              int64_t m, int64_t n, float *ef, uint8_t *codes, uint8_t *scales,
                              float *transformed);

/* Rank mean of MXFP4-encoded ranks: mean[e] = fl32(acc / N), acc = fl32(acc +
 * v_j[e]) for j = 0..N-1 in order, v_j = E2M1 value x 2^(scale - 127) (exact;
 * NaN for scale 255).  codes [N, m, n/2] (4-byte aligned), scales
 * [N, m, n/32], mean [m, n] float32 out (16-byte aligned); n % 32 == 0. */
gift_status gift_reduce_local_mxfp4(gift_ctx *ctx, const uint8_t *codes, const uint8_t *scales,
                                    int32_t N, int64_t m, int64_t n, float *mean);

/* Average the N ranks in transformed coordinates (eq. dp_grad_avg):
 *   mean[e] = fl32(acc / N),  acc = fl32(acc + fl32(val(codes[j][e]) * s_j)) for
 *   j = 0..N-1 in order (no fused multiply-add), s_j the scale of e's block.
 * Dequantizing each rank with its own scale is Algorithm 1's
 * Dequantize(AllReduce_SUM(Q); s) / N whenever the scales are shared.
 *   codes [N, m, n], scales [N, nbr, nbc], mean [m, n] float32 out. */
gift_status gift_reduce_local(gift_ctx *ctx, const uint8_t *codes, const float *scales,
                              int32_t N, int64_t m, int64_t n, int32_t block_rows,
                              int32_t block_cols, float *mean);

/* Inverse transform (eq. design_full_inverse_transform): out = S_G mean S_A
 * (sides absent from f are the identity; f = NULL copies).  mean and out are
 * [m, n] float32 and must not overlap. */
gift_status gift_decode(gift_ctx *ctx, const gift_factor *f, const float *mean,
                        int64_t m, int64_t n, float *out);

/* gift_decode of many matrices of one shape in one call (the inverse
 * transform of eq. design_input_side_inverse for every matrix of a gradient
 * bucket set, Algorithm 1's last step): out[i] = decode(factors[i], means[i]).
 * factors, means and outs are HOST arrays of count device handles /
 * pointers; every mean and out is [m, n] float32, outs distinct and not
 * aliasing their means.  When every factor is a low-rank input-side factor
 * of one rank r in {16, 32, 64, 128}, or every factor is a two-sided
 * low-rank factor with rank r in that set on both sides (eq.
 * design_full_inverse_transform), and the buffers are 16-byte aligned, each
 * pass (each product of the inverse) runs as one launch over all matrices
 * with the kernels, split-K partials and summation order of gift_decode, so
 * the results equal count separate gift_decode calls bit for bit; the
 * per-matrix operand pointers come from device tables the context uploads
 * (through its pinned buffer) only when they change.  Otherwise the call
 * runs count gift_decode calls.  Uses the context workspace (the
 * projections of all count matrices: count * parts * m * r floats, and for
 * two-sided factors also their Q, K and L2 terms).  Errors: as gift_decode;
 * GIFT_EINVAL for NULL arrays, a count outside [0, 65535] or an output
 * listed twice. */
gift_status gift_decode_batch(gift_ctx *ctx, int32_t count, const gift_factor *const *factors,
                              const float *const *means, float *const *outs, int64_t m, int64_t n);

#ifdef __cplusplus
}
#endif

#endif /* GIFT_H */
