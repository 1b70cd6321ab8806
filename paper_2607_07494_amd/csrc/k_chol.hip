// Cholesky-form transforms of the K-FAC factors (Sec. IV-A, eq. design_chol,
// eq. design_full_transform / design_input_side_transform and their inverses)
// and Table II's cheaper approximations of A: its diagonal (diag-A) and its
// b x b diagonal blocks (block-A-b).
//
// A side is refreshed from its statistics A = X^T X / T as the Cholesky
// factor of A + delta I, delta = damping * tr(A) / dim, restricted to b x b
// diagonal blocks (b = dim: the full factor).  Each block is factored in
// float64 by the Cholesky kernels of the subspace pipeline (which also write
// R = L_k^T), the diagonal variant by one elementwise kernel.
//
// The transforms are block-diagonal triangular products: the input side
// multiplies every rank's rows by blockdiag(R^-1) (forward, W L^-T) or
// blockdiag(R) (inverse, M L^T); the output side multiplies from the left by
// the transposed blocks (L^-1 W, L M).  They run on the float32 tile kernel
// with one batch entry per diagonal block (zero blocks are never touched);
// the diagonal variant is one elementwise pass.
#include <math.h>

#include "gift_internal.h"

namespace gift {
namespace {

constexpr int kShiftThreads = 256;

// shift[0] = damping * tr(A) / dim, shift[1] = tr(A); the trace in float64,
// every thread summing a fixed strided subset, then a fixed tree
__global__ __launch_bounds__(kShiftThreads) void chol_shift_kernel(const float *A, int64_t dim, float damping,
                                                                   float *shift) {
  __shared__ double part[kShiftThreads];
  double s = 0.0;
  for (int64_t i = threadIdx.x; i < dim; i += kShiftThreads) s += (double)A[i * dim + i];
  part[threadIdx.x] = s;
  __syncthreads();
  for (int w = kShiftThreads / 2; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double tr = part[0];
    shift[0] = (float)((double)damping * tr / (double)dim);
    shift[1] = (float)tr;
  }
}

// G[blk][i][j] = A_(blk b + i, blk b + j) + delta [i == j] inside the
// block's kv x kv part, the identity outside it; all identity when tr(A) <= 0
__global__ void chol_gather_kernel(const float *A, int64_t dim, int b, int64_t total, const float *shift,
                                   float *G) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= total) return;
  const int64_t bb = (int64_t)b * b;
  const int64_t blk = t / bb;
  const int64_t e = t - blk * bb;
  const int i = (int)(e / b), j = (int)(e - (int64_t)i * b);
  const int64_t r0 = blk * b;
  const int64_t kv = dim - r0 < b ? dim - r0 : b;
  const bool ident = !(shift[1] > 0.f) || i >= kv || j >= kv;
  float v;
  if (ident) v = i == j ? 1.f : 0.f;
  else v = A[(r0 + i) * dim + r0 + j] + (i == j ? shift[0] : 0.f);
  G[t] = v;
}

// 1 x 1 blocks: R = sqrt(g), R^-1 = 1 / sqrt(g), in float64
__global__ void chol_diag_kernel(const float *G, int64_t count, float *R, float *Rinv) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= count) return;
  const double g = (double)G[t];
  const double d = g > 0.0 ? g : 1e-300;
  const double r = sqrt(d);
  R[t] = (float)r;
  Rinv[t] = (float)(1.0 / r);
}

// y = x * rowscale[row] * colscale[col] over [N, m, n] (either scale may be absent)
__global__ void chol_scale_kernel(const float *x, float *y, int64_t m, int64_t n, int64_t total,
                                  const float *rowscale, const float *colscale) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= total) return;
  const int64_t rc = t / n;
  const int64_t c = t - rc * n;
  float v = x[t];
  if (rowscale) v *= rowscale[rc % m];
  if (colscale) v *= colscale[c];
  y[t] = v;
}

__global__ void chol_identity_kernel(float *R, float *Rinv, int b, int64_t total) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= total) return;
  const int64_t e = t % ((int64_t)b * b);
  const float v = (e / b == e % b) ? 1.f : 0.f;
  R[t] = v;
  Rinv[t] = v;
}

unsigned grid1(int64_t total, int threads) { return (unsigned)((total + threads - 1) / threads); }

// Y = X blockdiag(mats) for X, Y [rows, dim] (rows = ranks x rows per rank)
gift_status right_mul(gift_ctx *ctx, const CholSide &s, const float *mats, const float *X, float *Y,
                      int64_t rows) {
  const int64_t dim = s.dim, b = s.b;
  const int64_t nfull = dim / b, kv = dim - nfull * b;
  for (int part = 0; part < 2; ++part) {
    const int64_t cnt = part == 0 ? nfull : (kv > 0 ? 1 : 0);
    const int64_t w = part == 0 ? b : kv;
    if (cnt == 0) continue;
    const int64_t c0 = part == 0 ? 0 : nfull * b;
    TileJob j;
    j.nseg = 1;
    j.seg[0].a = Operand{X + c0, dim, b, true};          // (i, k) at X[i dim + blk b + k]
    j.seg[0].b = Operand{mats + (c0 / b) * b * b, b, b * b, false};   // (k, c) at blk[k][c]
    j.seg[0].K = w;
    j.M = rows;
    j.N = w;
    j.batch = (int32_t)cnt;
    j.C = Y + c0;
    j.ldc = dim;
    j.cbs = b;
    j.kernel_family = GIFT_KERNEL_CHOL_TRANSFORM;
    gift_status st = launch_tile(ctx, j);
    if (st != GIFT_OK) return st;
  }
  return GIFT_OK;
}

// Y_r = blockdiag(mats)^T X_r for every rank r, X, Y [N, dim, n]
gift_status left_mul_t(gift_ctx *ctx, const CholSide &s, const float *mats, const float *X, float *Y,
                       int32_t N, int64_t n) {
  const int64_t dim = s.dim, b = s.b;
  const int64_t nfull = dim / b, kv = dim - nfull * b;
  const int64_t per = dim * n;
  if (nfull == 1 && kv == 0) {   // the full factor: one launch over the ranks
    TileJob j;
    j.nseg = 1;
    j.seg[0].a = Operand{mats, b, 0, false};   // (i, k) = mats[k][i]
    j.seg[0].b = Operand{X, n, per, false};    // (k, c) = X_r[k][c]
    j.seg[0].K = b;
    j.M = b;
    j.N = n;
    j.batch = N;
    j.C = Y;
    j.ldc = n;
    j.cbs = per;
    j.kernel_family = GIFT_KERNEL_CHOL_TRANSFORM;
    return launch_tile(ctx, j);
  }
  for (int32_t r = 0; r < N; ++r) {
    for (int part = 0; part < 2; ++part) {
      const int64_t cnt = part == 0 ? nfull : (kv > 0 ? 1 : 0);
      const int64_t w = part == 0 ? b : kv;
      if (cnt == 0) continue;
      const int64_t r0 = part == 0 ? 0 : nfull * b;
      TileJob j;
      j.nseg = 1;
      j.seg[0].a = Operand{mats + (r0 / b) * b * b, b, b * b, false};
      j.seg[0].b = Operand{X + r * per + r0 * n, n, b * n, false};
      j.seg[0].K = w;
      j.M = w;
      j.N = n;
      j.batch = (int32_t)cnt;
      j.C = Y + r * per + r0 * n;
      j.ldc = n;
      j.cbs = b * n;
      j.kernel_family = GIFT_KERNEL_CHOL_TRANSFORM;
      gift_status st = launch_tile(ctx, j);
      if (st != GIFT_OK) return st;
    }
  }
  return GIFT_OK;
}

}  // namespace

gift_status chol_side_identity(gift_ctx *ctx, CholSide &s) {
  const int64_t total = (int64_t)s.nblk * s.b * s.b;
  ProfileScope prof(ctx, GIFT_KERNEL_SMALL);
  hipLaunchKernelGGL(chol_identity_kernel, dim3(grid1(total, 256)), dim3(256), 0, ctx->stream, s.R, s.Rinv,
                     s.b, total);
  return check_launch("chol_identity");
}

gift_status chol_side_update(gift_ctx *ctx, CholSide &s, const void *x, int64_t T, gift_dtype dtype,
                             float damping) {
  const int64_t dim = s.dim;
  // statistics A = X^T X / T into the side's own buffer
  const bool widen = dtype == GIFT_BF16 && !statistics_direct(dtype, dim);
  void *ws = nullptr;
  gift_status st = workspace(ctx, widen ? sizeof(float) * (size_t)T * dim : 256, &ws);
  if (st != GIFT_OK) return st;
  float *Xc = widen ? static_cast<float *>(ws) : nullptr;
  void *d_tab = nullptr;
  if ((st = upload_table(ctx, TAB_CHOL_STATS, &s, &x, sizeof(void *), &d_tab)) != GIFT_OK) return st;
  if ((st = launch_statistics(ctx, static_cast<const void *const *>(d_tab), &x, 1, T, dim, dtype, s.A, Xc)) !=
      GIFT_OK)
    return st;
  {
    ProfileScope prof(ctx, GIFT_KERNEL_SMALL);
    hipLaunchKernelGGL(chol_shift_kernel, dim3(1), dim3(kShiftThreads), 0, ctx->stream, s.A, dim, damping,
                       s.shift);
    if ((st = check_launch("chol_shift")) != GIFT_OK) return st;
  }
  // the diagonal blocks of A + delta I, then their factors (a later
  // workspace growth synchronizes the stream first, so the statistics'
  // pointer table is no longer in use)
  const int64_t total = (int64_t)s.nblk * s.b * s.b;
  const size_t g_bytes = (sizeof(float) * (size_t)total + 255) & ~(size_t)255;
  const size_t scratch = s.b > 1 ? chol_blocks_scratch(s.b, s.nblk) : 0;
  if ((st = workspace(ctx, g_bytes + scratch, &ws)) != GIFT_OK) return st;
  float *G = static_cast<float *>(ws);
  {
    ProfileScope prof(ctx, GIFT_KERNEL_SMALL);
    hipLaunchKernelGGL(chol_gather_kernel, dim3(grid1(total, 256)), dim3(256), 0, ctx->stream, s.A, dim, s.b,
                       total, s.shift, G);
    if ((st = check_launch("chol_gather")) != GIFT_OK) return st;
  }
  if (s.b == 1) {
    ProfileScope prof(ctx, GIFT_KERNEL_CHOL);
    hipLaunchKernelGGL(chol_diag_kernel, dim3(grid1(total, 256)), dim3(256), 0, ctx->stream, G, total, s.R,
                       s.Rinv);
    return check_launch("chol_diag");
  }
  return launch_chol_blocks(ctx, G, s.b, s.nblk, s.R, s.Rinv, static_cast<char *>(ws) + g_bytes);
}

bool chol_transform_needs_tmp(const gift_factor *f) {
  const bool useA = f->CA.b > 0, useG = f->CG.b > 0;
  return useA && useG && !(f->CA.b == 1 && f->CG.b == 1);
}

gift_status launch_chol_transform(gift_ctx *ctx, const gift_factor *f, const float *in, float *out,
                                  int32_t N, bool inverse, float *tmp) {
  const int64_t m = f->m, n = f->n;
  const CholSide &A = f->CA, &G = f->CG;
  const bool useA = A.b > 0, useG = G.b > 0;
  const int64_t total = (int64_t)N * m * n;
  const float *mA = useA ? (inverse ? A.R : A.Rinv) : nullptr;
  const float *mG = useG ? (inverse ? G.R : G.Rinv) : nullptr;
  // diagonal factors: one elementwise pass covers both sides
  const bool dA = useA && A.b == 1, dG = useG && G.b == 1;
  if ((dA || !useA) && (dG || !useG)) {
    if (!useA && !useG) return launch_copy_f32(ctx, out, in, total);
    ProfileScope prof(ctx, GIFT_KERNEL_CHOL_TRANSFORM);
    hipLaunchKernelGGL(chol_scale_kernel, dim3(grid1(total, 256)), dim3(256), 0, ctx->stream, in, out, m, n,
                       total, mG, mA);
    return check_launch("chol_scale");
  }
  if (useA && useG) {   // two products through the caller's intermediate
    gift_status st = right_mul(ctx, A, mA, in, tmp, (int64_t)N * m);
    if (st != GIFT_OK) return st;
    return left_mul_t(ctx, G, mG, tmp, out, N, n);
  }
  if (useA) return right_mul(ctx, A, mA, in, out, (int64_t)N * m);
  return left_mul_t(ctx, G, mG, in, out, N, n);
}

}  // namespace gift
