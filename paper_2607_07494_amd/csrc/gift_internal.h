// Internal declarations of the GIFT codec library (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <map>
#include <string>
#include <utility>
#include <vector>

#include "gift.h"

namespace gift {

// ---------------------------------------------------------------------------
// Error reporting
// ---------------------------------------------------------------------------
gift_status set_error(gift_status st, const std::string &msg);
gift_status hip_error(hipError_t e, const char *what);

#define GIFT_HIP_TRY(expr)                                  \
  do {                                                      \
    hipError_t _e = (expr);                                 \
    if (_e != hipSuccess) return ::gift::hip_error(_e, #expr); \
  } while (0)

// ---------------------------------------------------------------------------
// Context and factor state
// ---------------------------------------------------------------------------
struct Workspace {
  void *ptr = nullptr;
  size_t bytes = 0;
};

struct ProfileRec {
  int kernel;
  hipEvent_t start, stop;
};

// A small device table (pointer and job tables of a launch sequence) with
// the host image it was last uploaded from.  Uploads go through pinned host
// memory owned by the context and happen only when the contents change, so
// a compute call with unchanged tables makes no host-to-device copy.
struct TableSlot {
  Workspace dev;
  void *pinned = nullptr;
  size_t pinned_bytes = 0;
  std::vector<char> last;
  hipEvent_t copied = nullptr;   // the last copy out of `pinned`
  bool valid = false;
};
enum TableKind { TAB_REFRESH = 0, TAB_STATS = 1, TAB_CHOL_STATS = 2, TAB_CHOL_BLOCKS = 3, TAB_DECODE = 4,
                 TAB_DECODE_BOTH = 5 };

// Per-matrix operands of a grouped decode (one batch entry per matrix): the
// rank mean, the factor's U^T and U diag(c'), and the output.
struct DecodePtrs {
  const float *mean;
  const float *ut;
  const float *uci;
  float *out;
};

}  // namespace gift

struct gift_ctx {
  hipStream_t stream = nullptr;
  int device = -1;                 // bound at the first compute call
  gift::Workspace ws;              // grow-only device workspace
  // Block-amax sub-slots: two sets used by alternate encodes.  The set an
  // encode starts with is all zero; the kernel that consumes a set's maxima
  // also clears what the previous encode left in the other set.
  gift::Workspace slots;
  gift::Workspace xform;           // transformed copies of the Cholesky-form transforms
  size_t slot_words = 0;           // capacity of one set
  int slot_set = 0;                // set of the next encode
  size_t slot_dirty[2] = {0, 0};   // words of each set still to clear
  bool slots_unknown = false;      // an encode stopped between its passes
  hipEvent_t stats_event = nullptr;  // caller's event, recorded after each refresh's statistics
  bool profile = false;
  uint32_t profile_mask = ~0u;     // kernel families timed when profiling
  std::vector<gift::ProfileRec> prof;
  int64_t prof_launches[GIFT_KERNEL_COUNT] = {};
  double prof_ms[GIFT_KERNEL_COUNT] = {};
  std::vector<hipEvent_t> event_pool;
  // set for the duration of an allocation-free call: no profiling events
  // are created or recorded
  bool no_alloc_call = false;
  // device tables by (kind, owner), see TableSlot
  std::map<std::pair<int, const void *>, gift::TableSlot> tables;
};

namespace gift {

// One side's transform S^-1 = I + U diag(c) U^T, kept in the layouts the
// kernels read with unit stride along the contraction index.
struct Side {
  int64_t dim = 0;       // n for the input side, m for the output side
  int32_t r = 0;
  int32_t k = 0;         // subspace block width (min(dim, 2r))
  float *Ut = nullptr;   // [r, dim]   U^T (rows = eigenvectors)
  float *U = nullptr;    // [dim, r]   U
  float *Uc = nullptr;   // [dim, r]   U diag(c_fwd)
  float *Uci = nullptr;  // [dim, r]   U diag(c_inv)
  float *c_fwd = nullptr, *c_inv = nullptr;   // [r]
  float *sigma2 = nullptr;                    // [1]
  float *lam = nullptr;                       // [r]
  float *Qt = nullptr;   // [k, dim]   warm-start block (rows orthonormal)
  bool have_basis = false;  // Qt holds a previous subspace
  bool fill_tail = false;   // Qt rows r..k-1 still need start-block rows
};

// One side's Cholesky-form transform: A + delta I ~ L L^T with L
// block-diagonal (b x b blocks; b = dim is the full factor, b = 1 the
// diagonal), stored per block as R = L_k^T and R^-1 (upper triangular,
// [nblk][b][b]; the last block's kv x kv part top-left, identity elsewhere).
struct CholSide {
  int64_t dim = 0;
  int32_t b = 0;          // 0: side absent
  int32_t nblk = 0;
  float *R = nullptr;
  float *Rinv = nullptr;
  float *A = nullptr;     // [dim, dim] statistics of the last update
  float *shift = nullptr; // [2]: delta, tr(A)
};

}  // namespace gift

struct gift_factor {
  gift_ctx *ctx = nullptr;
  int64_t m = 0, n = 0;
  int32_t rank = 0, sides = 0;
  float damping = 0.f;
  uint64_t seed = 0;
  gift::Side A;   // input side (dim n)
  gift::Side G;   // output side (dim m)
  bool chol = false;    // Cholesky-form factor (CA / CG) instead of the low-rank one
  int32_t block = 0;    // requested block size of a Cholesky-form factor
  gift::CholSide CA, CG;
  void *alloc = nullptr;
};

namespace gift {

// ---------------------------------------------------------------------------
// Launch plumbing
// ---------------------------------------------------------------------------
gift_status bind_device(gift_ctx *ctx);
// Device scratch of at least `bytes`, 256-byte aligned; may reallocate (and
// synchronize the stream) when it grows.
gift_status workspace(gift_ctx *ctx, size_t bytes, void **out);
// Bracket launches of one kernel family with events when profiling is on.
struct ProfileScope {
  gift_ctx *ctx;
  int kernel;
  hipEvent_t stop = nullptr;
  ProfileScope(gift_ctx *c, int k);
  ~ProfileScope();
};
gift_status check_launch(const char *what);

// ---------------------------------------------------------------------------
// Block geometry of the scale grid
// ---------------------------------------------------------------------------
struct BlockGeom {
  int64_t br, bc;      // block extent in rows / cols
  int32_t nbr, nbc;    // blocks per column / row
};
BlockGeom block_geom(int64_t m, int64_t n, int32_t block_rows, int32_t block_cols);

// ---------------------------------------------------------------------------
// Kernel launchers (enqueue on ctx->stream; no validation beyond asserts)
// ---------------------------------------------------------------------------

// Strided fp32 operand: element (i, k) of A at ptr[b*bs + i*ld + k] when
// kmajor, else ptr[b*bs + k*ld + i]; element (k, j) of B at
// ptr[b*bs + j*ld + k] when kmajor, else ptr[b*bs + k*ld + j].
struct Operand {
  const float *ptr = nullptr;
  int64_t ld = 0;
  int64_t bs = 0;
  bool kmajor = true;
  // the operand is the sum of `parts` split-K partials, partial z of batch b
  // at ptr + (b * parts + z) * bs (register-direct update kernel only)
  int parts = 1;
  // grouped decode of many matrices: batch entry b's operand starts at
  // tab[b] (device array; ptr and bs unused).  Taken by the tile kernel and
  // the register-direct update kernel only (job_has_tabs).
  const float *const *tab = nullptr;
};

struct Segment {
  Operand a, b;
  int64_t K = 0;
};

enum Epilogue { EPI_STORE = 0, EPI_AMAX = 1, EPI_QUANT = 2, EPI_MX = 3 };

// Block maxima are accumulated with atomicMax into kAmaxSlots sub-slots per
// (rank, block) -- producers pick a slot from their wave id, so no single
// address sees more than a few atomics -- and finalize_amax reduces the slots
// (and the ranks, for a shared scale) into one value per (rank, block).
constexpr int kAmaxSlots = 64;

struct TileJob {
  // C = sum_s A_s B_s over up to two segments (nseg = 0: no product)
  Segment seg[2];
  int nseg = 0;
  int64_t M = 0, N = 0;     // output rows / cols
  int32_t batch = 1;
  int32_t ksplit = 1;         // STORE only: partial sums to C + (b*ksplit+s)*cbs
  // STORE: C = (alpha*acc + beta*D) * colscale[j]
  float *C = nullptr;
  int64_t ldc = 0, cbs = 0;
  const float *D = nullptr;  // addend (required for the codec epilogues)
  int64_t ldd = 0, dbs = 0;
  float alpha = 1.f, beta = 0.f;
  const float *colscale = nullptr;
  // codec epilogues (W~ = D + acc [+ R]); matrices are [batch, M, N] dense
  // amax: AMAX pass -> raw slots [batch, nbr, nbc, kAmaxSlots] (atomicMax of
  //       float bits); QUANT pass -> finished values [batch, nbr, nbc]
  uint32_t *amax = nullptr;
  uint8_t *codes = nullptr;
  uint32_t *hits = nullptr;   // QUANT: boundary-hit counters [batch][2] (upper, lower), accumulated
  // MXFP4 in the update pass (split-bf16 kernel only): packed codes
  // [batch][M][N/2] and E8M0 scales [batch][M][N/32]; amax stays null
  uint8_t *mx_codes = nullptr;
  uint8_t *mx_scales = nullptr;
  float *scales = nullptr;
  float *transformed = nullptr;
  float *ef = nullptr;
  bool ef_added = false;     // D already holds W~ + R (quantize a stored W~)
  // QUANT pass of the streaming kernel straight from the AMAX pass's raw
  // sub-slots (amax = raw): block maxima and scales in the kernel, and
  // clear_words words at clear zeroed
  bool from_raw = false;
  uint32_t *clear = nullptr;
  int64_t clear_words = 0;
  BlockGeom geom{};
  bool shared = false;
  // form the products from bf16 hi/lo splits of both operands on the bf16
  // matrix cores (k_lowrank.hip) where the shapes allow; float32 otherwise
  bool split3 = false;
  int kernel_family = GIFT_KERNEL_FACTOR;
  // grouped decode (k_update.hip kernels only): batch entry b takes its
  // mean / U^T (projection) and U diag(c') / mean / output (update) from
  // decode_tab[b] (device) instead of base + b * stride
  const DecodePtrs *decode_tab = nullptr;
  // the encode's update: each segment's column operand split into bf16 hi /
  // lo fragments in the LDS layout of its 64-column tiles
  // (launch_lr_col_image), which the sweep variant copies straight into LDS;
  // img_bs / img_bs2: bytes between batch entries' images (0: shared)
  const void *col_img = nullptr;
  const void *col_img2 = nullptr;
  int64_t img_bs = 0, img_bs2 = 0;
  // grouped decode: per-entry column scales (tile kernel), addend and output
  // (update kernel), device arrays indexed by the batch entry
  const float *const *colscale_tab = nullptr;
  const float *const *d_tab = nullptr;
  float *const *c_tab = nullptr;
  // the two-sided AMAX pass at rank 96 or 128 stores W~ to `transformed` in
  // the sweep variant (the encode then quantizes the stored W~)
  bool sweep_store = false;
};

gift_status launch_tile(gift_ctx *ctx, const TileJob &job);
// the job reaches some operand, addend, output or column scale through a
// per-entry pointer table
inline bool job_has_tabs(const TileJob &j) {
  for (int s = 0; s < j.nseg && s < 2; ++s)
    if (j.seg[s].a.tab || j.seg[s].b.tab) return true;
  return j.colscale_tab || j.d_tab || j.c_tab;
}
// k_lowrank.hip: the encode's projection and rank-r update with split bf16
// operands; lr_proj_parts = split-K partials of the projection
bool lr_update_eligible(const TileJob &job);
// its quantize pass can take the AMAX pass's raw sub-slots (job.from_raw)
bool lr_quant_reads_raw(const TileJob &job);
gift_status launch_lr_update(gift_ctx *ctx, const TileJob &job);
bool lr_proj_eligible(const TileJob &job);
gift_status launch_lr_proj(gift_ctx *ctx, const TileJob &job);
int lr_proj_parts(int64_t M, int64_t K, int32_t batch);
// the encode's output-side projection Q^T = W^T U_G with split bf16
// operands (job: A = W read transposed, B = U^T k-major and shared, r = 64
// or 128, M a multiple of 64): lr_projT_parts = its split-K partial count
// for the shape (0: not this kernel), which the job's ksplit must equal
int lr_projT_parts(int64_t M, int64_t K, int64_t r, int32_t batch);
bool lr_projT_eligible(const TileJob &job);
gift_status launch_lr_projT(gift_ctx *ctx, const TileJob &job);
// the column-operand image of the encode's sweep update: col [N][K] (row
// stride ld) -> bf16 hi / lo fragments of each 64-column tile, K = 64, 96 or
// 128 and N a multiple of 128; lr_col_image_bytes = its size (0: no image
// for this shape).  count > 1: count operands col_bs floats apart, their
// images lr_col_image_bytes apart
size_t lr_col_image_bytes(int64_t N, int K);
gift_status launch_lr_col_image(gift_ctx *ctx, const float *col, int64_t ld, int64_t N, int K, void *img,
                                int32_t count = 1, int64_t col_bs = 0);
// out[b] = sum_z partials[b][z] (in order) for [batch][parts][per_rank] floats
// (per_rank a multiple of 4, 16-byte aligned buffers)
gift_status launch_lr_psum(gift_ctx *ctx, const float *partials, float *out, int parts, int64_t per_rank,
                           int32_t batch, int kernel_family);
// k_update.hip: register-direct rank-r update / projection (used by
// launch_tile when the job's shapes allow)
bool update_kernel_eligible(const TileJob &job);
gift_status launch_update(gift_ctx *ctx, const TileJob &job);
bool proj_kernel_eligible(const TileJob &job);
// launch_proj takes the LDS-staged projection kernel (the one that reads a
// grouped decode's table) for this job
bool proj_staged_eligible(const TileJob &job);
// k_stream.hip: streaming Euclidean amax / quantize and rank sum
bool stream_eligible(int64_t m, int64_t n, const BlockGeom &g, const void *x, const void *codes,
                     const void *a, const void *b);
gift_status launch_stream_codec(gift_ctx *ctx, const TileJob &job);
gift_status launch_stream_reduce(gift_ctx *ctx, const uint8_t *codes, const float *scales, int32_t N,
                                 int64_t m, int64_t n, BlockGeom g, float *mean);
gift_status launch_proj(gift_ctx *ctx, const TileJob &job);
// split-K factor the projection kernel uses for an [batch, M, K] x [C, K]^T
// product whose consumer can sum partials (1 = a single result)
int proj_parts(int64_t M, int64_t K, int C, int32_t batch);
gift_status launch_zero_u32(gift_ctx *ctx, uint32_t *p, int64_t count);
// raw [N, nblk, kAmaxSlots] -> final [N, nblk] (max over slots, and over ranks
// when shared) and scales s = amax / 448; clears the raw slots it read and
// `clear_words` words at `clear`
gift_status launch_finalize_amax(gift_ctx *ctx, uint32_t *raw, int32_t N, int64_t nblk,
                                 bool shared, uint32_t *final_amax, float *scales, uint32_t *clear,
                                 int64_t clear_words);
// Sub-slot set for an encode that needs `words` words: *cur (all zero) and the
// other set with the words it still holds from the previous encode (to be
// cleared by this encode's last kernel).  Grows both sets on demand.
gift_status amax_slots(gift_ctx *ctx, size_t words, uint32_t **cur, uint32_t **other,
                       size_t *other_dirty);
// Book-keeping after this encode's last kernel: the current set holds
// `left` words (0 if its consumer cleared it), the other set is clean.
void amax_slots_done(gift_ctx *ctx, size_t left);
gift_status launch_reduce(gift_ctx *ctx, const uint8_t *codes, const float *scales,
                          int32_t N, int64_t m, int64_t n, BlockGeom g, float *mean);
gift_status launch_copy_f32(gift_ctx *ctx, float *dst, const float *src, int64_t count);

// factor pipeline (k_factor.hip): sides with equal (dim, r) are refreshed
// together in one launch sequence
struct SideJob {
  Side *side;
  const void *x;      // [T, dim] statistics input (device)
  uint64_t seed;      // Philox key of the start block
  float damping;
};
// A_m = X_m^T X_m / T for G inputs of one dimension into A [G, dim, dim]:
// bf16 inputs with dim % 8 == 0 on the bf16 SYRK kernel (device pointer table
// d_xtab), otherwise the float32 tile kernel (host pointers h_x; bf16 inputs
// are widened into Xc [T, dim] first).
bool statistics_direct(gift_dtype dtype, int64_t dim);
gift_status launch_statistics(gift_ctx *ctx, const void *const *d_xtab, const void *const *h_x, int G,
                              int64_t T, int64_t dim, gift_dtype dtype, float *A, float *Xc);
gift_status factor_refresh_batch(gift_ctx *ctx, const std::vector<SideJob> &jobs, int64_t T,
                                 gift_dtype dtype, int32_t iters);
gift_status side_import(gift_ctx *ctx, Side &s, const float *U, const float *c_fwd,
                        const float *c_inv, const float *sigma2);
gift_status side_export(gift_ctx *ctx, const Side &s, float *U, float *c_fwd,
                        float *c_inv, float *sigma2);
gift_status side_set_identity(gift_ctx *ctx, Side &s);

// k_factor.hip: Cholesky and inverse of `count` k x k blocks G (contiguous
// [count][k][k], symmetric positive definite): R [count][k][k] with
// G = R^T R (upper triangular) and Rinv = R^-1, float64 inside.  `scratch`
// holds chol_blocks_scratch(k, count) bytes of device memory.
size_t chol_blocks_scratch(int k, int count);
gift_status launch_chol_blocks(gift_ctx *ctx, const float *G, int k, int count, float *R, float *Rinv,
                               void *scratch);

// k_chol.hip: Cholesky-form factors and transforms
// Refresh one side from its [T, dim] statistics input.
gift_status chol_side_update(gift_ctx *ctx, CholSide &s, const void *x, int64_t T, gift_dtype dtype,
                             float damping);
// Identity transform (R = R^-1 = I).
gift_status chol_side_identity(gift_ctx *ctx, CholSide &s);
// out[N, m, n] = L_G^-1 in L_A^-T (forward) or L_G in L_A^T (inverse) for the
// sides the factor has; in and out must not overlap.  tmp: [N, m, n] floats
// when chol_transform_needs_tmp(f) (two sides, not both diagonal), else unused.
bool chol_transform_needs_tmp(const gift_factor *f);
gift_status launch_chol_transform(gift_ctx *ctx, const gift_factor *f, const float *in, float *out,
                                  int32_t N, bool inverse, float *tmp);
// k_mx.hip: MXFP4 (OCP MX: E2M1 elements, E8M0 scale per 32 elements of a row)
// encode of x (+ ef_in) into packed codes [total / 2] and scales [total / 32]
// (total a multiple of 32, x / ef / transformed 16-byte aligned, codes 4-byte
// aligned), and the rank mean of N such ranks of per_rank elements each.
gift_status launch_mx_quant(gift_ctx *ctx, const float *x, const float *ef_in, float *ef, float *transformed,
                            uint8_t *codes, uint8_t *scales, int64_t total);
gift_status launch_mx_reduce(gift_ctx *ctx, const uint8_t *codes, const uint8_t *scales, int32_t N,
                             int64_t per_rank, float *mean);
// Grow-only device buffer (synchronizes the stream before it frees the old one).
gift_status grow_buffer(gift_ctx *ctx, Workspace &w, size_t bytes, void **out);
// Device copy of a small host table for (kind, owner): the cached copy when
// the bytes equal the last upload, else an asynchronous upload through the
// context's pinned buffer (waiting first for that buffer's previous copy).
gift_status upload_table(gift_ctx *ctx, int kind, const void *owner, const void *host, size_t bytes,
                         void **dev);

}  // namespace gift
