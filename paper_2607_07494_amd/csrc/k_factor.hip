// Factor refresh: K-FAC statistics and their rank-r transform.
//
// A = X^T X / T (eq. kfac_fisher_block, eq. impl_A_psd), then its leading r
// eigenpairs (eq. impl_A_lowrank) by block subspace iteration with
// k = min(dim, 2r) columns:
//
//   Q <- CholQR2(start);  repeat iters: Q <- CholQR2(A Q)
//   B = Q^T A Q;  B = V diag(theta) V^T (theta descending);  U = Q V[:, :r]
//
// (Golub & Van Loan, Matrix Computations, Sec. 8.2.4 and 8.1.6; CholeskyQR2
// after Fukaya et al. 2014.)  The dense products run on the tile kernel's
// FP32 MFMA path; the k x k steps (Cholesky, triangular inverse, symmetric
// eigensolver) are small single-workgroup kernels in float64.  The
// eigensolver is one-sided (Hestenes) Jacobi with round-robin parallel
// ordering: rotating the columns of the symmetric positive semidefinite B
// until they are mutually orthogonal yields B V = V diag(theta), so column
// norms are the eigenvalues and normalised columns the eigenvectors.
//
// The isotropic level and the coefficients follow the low-rank transform
// S^-1 = I + U diag(c) U^T with c_i = sqrt(sigma^2/lambda_i) - 1 and
// S = I + U diag(c') U^T with c'_i = sqrt(lambda_i/sigma^2) - 1, sigma^2 the
// mean of the discarded eigenvalues (floored at damping * tr(A)/dim).
//
// The start block is Philox4x32-10 (Salmon et al., SC'11): entry (i, j) is
// word 0 of the generator at counter (i, j, 0, 0), key (seed lo, seed hi),
// read as int32, shifted right by 8 and scaled by 2^-23.

#include <math.h>

#include "gift_internal.h"

namespace gift {

namespace {

constexpr int kSmallThreads = 1024;

__device__ __forceinline__ uint32_t philox_word0(uint32_t c0, uint32_t c1, uint32_t c2,
                                                 uint32_t c3, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint64_t p0 = (uint64_t)0xD2511F53u * c0;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
    const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    const uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  return c0;
}

// Qt[j][i] for rows j in [row0, k): the start block transposed.
__global__ void start_block_kernel(float *Qt, int64_t dim, int k, int row0, uint32_t k0,
                                   uint32_t k1) {
  const int64_t total = (int64_t)(k - row0) * dim;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int j = row0 + (int)(t / dim);
    const int64_t i = t % dim;
    const uint32_t w = philox_word0((uint32_t)i, (uint32_t)j, 0u, 0u, k0, k1);
    Qt[(int64_t)j * dim + i] = (float)(((int32_t)w) >> 8) * 1.1920928955078125e-7f;
  }
}

__global__ void bf16_to_f32_kernel(float *dst, const uint16_t *src, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = __uint_as_float((uint32_t)src[i] << 16);
}

// Sum split-K partials [ks][k][k] (float32) into W (float64, k x k).
__device__ void sum_partials(double *W, const float *part, int ks, int k) {
  const int64_t kk = (int64_t)k * k;
  for (int64_t t = threadIdx.x; t < kk; t += blockDim.x) {
    double s = 0.0;
    for (int z = 0; z < ks; ++z) s += (double)part[z * kk + t];
    W[t] = s;
  }
}

__device__ double block_sum(double v, double *red) {
  const int tid = threadIdx.x;
  red[tid] = v;
  __syncthreads();
  for (int s = blockDim.x / 2; s > 0; s >>= 1) {
    if (tid < s) red[tid] += red[tid + s];
    __syncthreads();
  }
  const double r = red[0];
  __syncthreads();
  return r;
}

// Gram partials -> R (upper Cholesky, pivots floored) -> Rinv (float32).
// W and X are float64 k x k scratch.
__global__ __launch_bounds__(kSmallThreads) void chol_inv_kernel(const float *part, int ks, int k,
                                                                 double *W, double *X,
                                                                 float *Rinv) {
  __shared__ double red[kSmallThreads];
  const int tid = threadIdx.x, nt = blockDim.x;
  sum_partials(W, part, ks, k);
  __syncthreads();
  double tr = 0.0;
  for (int i = tid; i < k; i += nt) tr += W[(int64_t)i * k + i];
  tr = block_sum(tr, red);
  const double floor = 1e-12 * (tr > 0.0 ? tr : 0.0) / (k > 0 ? k : 1) + 1e-300;
  // right-looking Cholesky on the upper triangle: W <- R
  for (int j = 0; j < k; ++j) {
    if (tid == 0) {
      const double d = W[(int64_t)j * k + j];
      W[(int64_t)j * k + j] = sqrt(d > floor ? d : floor);
    }
    __syncthreads();
    const double rjj = W[(int64_t)j * k + j];
    for (int l = j + 1 + tid; l < k; l += nt) W[(int64_t)j * k + l] /= rjj;
    __syncthreads();
    const int rem = k - j - 1;
    for (int64_t t = tid; t < (int64_t)rem * rem; t += nt) {
      const int a = j + 1 + (int)(t / rem), b = j + 1 + (int)(t % rem);
      if (b >= a) W[(int64_t)a * k + b] -= W[(int64_t)j * k + a] * W[(int64_t)j * k + b];
    }
    __syncthreads();
  }
  // X = R^-1 (upper), row by row from the bottom; columns in parallel
  for (int i = k - 1; i >= 0; --i) {
    const double rii = W[(int64_t)i * k + i];
    for (int c = tid; c < k; c += nt) {
      double v;
      if (c < i) {
        v = 0.0;
      } else if (c == i) {
        v = 1.0 / rii;
      } else {
        double s = 0.0;
        for (int l = i + 1; l <= c; ++l) s += W[(int64_t)i * k + l] * X[(int64_t)l * k + c];
        v = -s / rii;
      }
      X[(int64_t)i * k + c] = v;
    }
    __syncthreads();
  }
  for (int64_t t = tid; t < (int64_t)k * k; t += nt) Rinv[t] = (float)X[t];
}

// Rayleigh-Ritz: B partials -> eigenpairs by one-sided Jacobi -> top r.
// W: float64 k x k scratch (column-major working copy: W[c*k + row]),
// theta: float64 [k] out (sorted, top r), Vr: float32 [k][r] out.
__global__ __launch_bounds__(kSmallThreads) void rr_eig_kernel(const float *part, int ks, int k,
                                                               int r, double *W, double *norms,
                                                               double *theta, float *Vr,
                                                               int max_sweeps) {
  __shared__ double red[kSmallThreads];
  __shared__ int pair_p[512], pair_q[512];
  __shared__ double rot_c[512], rot_s[512];
  __shared__ int any_rot;
  const int tid = threadIdx.x, nt = blockDim.x;
  const int64_t kk = (int64_t)k * k;
  // symmetrised B, stored column-major (columns are the rotated vectors)
  for (int64_t t = tid; t < kk; t += nt) {
    const int i = (int)(t / k), j = (int)(t % k);
    double a = 0.0, b = 0.0;
    for (int z = 0; z < ks; ++z) {
      a += (double)part[z * kk + (int64_t)i * k + j];
      b += (double)part[z * kk + (int64_t)j * k + i];
    }
    W[(int64_t)j * k + i] = 0.5 * (a + b);
  }
  __syncthreads();
  const int kp = (k + 1) & ~1;  // players (one dummy when k is odd)
  const int npairs = kp / 2;
  for (int sweep = 0; sweep < max_sweeps; ++sweep) {
    if (tid == 0) any_rot = 0;
    __syncthreads();
    for (int round = 0; round < kp - 1; ++round) {
      // circle method: player kp-1 fixed, the others rotate
      for (int pi = tid; pi < npairs; pi += nt) {
        int p, q;
        if (pi == 0) {
          p = round;
          q = kp - 1;
        } else {
          p = (round + pi) % (kp - 1);
          q = (round - pi + kp - 1) % (kp - 1);
        }
        if (p > q) {
          const int t = p;
          p = q;
          q = t;
        }
        pair_p[pi] = p;
        pair_q[pi] = q;
      }
      __syncthreads();
      // rotation per pair from the column dot products
      for (int pi = tid; pi < npairs; pi += nt) {
        const int p = pair_p[pi], q = pair_q[pi];
        double c = 1.0, s = 0.0;
        if (q < k) {
          const double *cp = W + (int64_t)p * k, *cq = W + (int64_t)q * k;
          double alpha = 0.0, beta = 0.0, gamma = 0.0;
          for (int i = 0; i < k; ++i) {
            alpha += cp[i] * cp[i];
            beta += cq[i] * cq[i];
            gamma += cp[i] * cq[i];
          }
          if (fabs(gamma) > 1e-12 * sqrt(alpha * beta) && gamma != 0.0) {
            const double zeta = (beta - alpha) / (2.0 * gamma);
            const double t = (zeta >= 0.0 ? 1.0 : -1.0) / (fabs(zeta) + sqrt(1.0 + zeta * zeta));
            c = 1.0 / sqrt(1.0 + t * t);
            s = c * t;
            any_rot = 1;
          }
        }
        rot_c[pi] = c;
        rot_s[pi] = s;
      }
      __syncthreads();
      for (int64_t t = tid; t < (int64_t)npairs * k; t += nt) {
        const int pi = (int)(t / k), i = (int)(t % k);
        const int p = pair_p[pi], q = pair_q[pi];
        if (q >= k) continue;
        const double c = rot_c[pi], s = rot_s[pi];
        if (s == 0.0) continue;
        double *cp = W + (int64_t)p * k, *cq = W + (int64_t)q * k;
        const double a = cp[i], b = cq[i];
        cp[i] = c * a - s * b;
        cq[i] = s * a + c * b;
      }
      __syncthreads();
    }
    if (!any_rot) break;
    __syncthreads();
  }
  // eigenvalue = column norm, eigenvector = column / norm
  for (int j = tid; j < k; j += nt) {
    double s = 0.0;
    for (int i = 0; i < k; ++i) s += W[(int64_t)j * k + i] * W[(int64_t)j * k + i];
    norms[j] = sqrt(s);
  }
  __syncthreads();
  // rank columns by descending eigenvalue (ties by index), keep the top r
  for (int j = tid; j < k; j += nt) {
    const double v = norms[j];
    int rank = 0;
    for (int l = 0; l < k; ++l) {
      const double u = norms[l];
      rank += (u > v) || (u == v && l < j);
    }
    if (rank < r) {
      theta[rank] = v;
      const double inv = v > 0.0 ? 1.0 / v : 0.0;
      for (int i = 0; i < k; ++i) Vr[(int64_t)i * r + rank] = (float)(W[(int64_t)j * k + i] * inv);
    }
  }
}

// sigma^2, coefficients and the U layouts from Ut and theta.
__global__ __launch_bounds__(kSmallThreads) void finalize_kernel(
    const float *Amat, int64_t dim, const double *theta, int r, float damping, const float *Ut,
    float *U, float *Uc, float *Uci, float *c_fwd, float *c_inv, float *lam_out, float *sigma2_out,
    double *scratch) {
  __shared__ double red[kSmallThreads];
  const int tid = threadIdx.x, nt = blockDim.x;
  double tr = 0.0;
  for (int64_t i = tid; i < dim; i += nt) tr += (double)Amat[i * dim + i];
  tr = block_sum(tr, red);
  double top = 0.0;
  for (int i = tid; i < r; i += nt) top += theta[i] > 0.0 ? theta[i] : 0.0;
  top = block_sum(top, red);
  double sigma2 = 0.0;
  const bool identity = !(tr > 0.0) || r == 0;
  const double floor = (double)damping * tr / (double)dim;
  if (!identity) {
    if (r >= dim) {
      sigma2 = tr / (double)dim;
    } else {
      sigma2 = (tr - top) / (double)(dim - r);
      if (sigma2 < floor) sigma2 = floor;
    }
  }
  for (int i = tid; i < r; i += nt) {
    double l = theta[i] > 0.0 ? theta[i] : 0.0;
    double cf = 0.0, ci = 0.0;
    if (!identity) {
      const double fl = r >= dim ? floor : sigma2;
      if (l < fl) l = fl;
      cf = sqrt(sigma2 / l) - 1.0;
      ci = sqrt(l / sigma2) - 1.0;
    }
    scratch[2 * i] = cf;
    scratch[2 * i + 1] = ci;
    c_fwd[i] = (float)cf;
    c_inv[i] = (float)ci;
    lam_out[i] = (float)l;
  }
  if (tid == 0) sigma2_out[0] = (float)sigma2;
  __syncthreads();
  for (int64_t t = tid; t < dim * r; t += nt) {
    const int64_t i = t / r;
    const int a = (int)(t % r);
    const float u = Ut[(int64_t)a * dim + i];
    U[t] = u;
    Uc[t] = (float)((double)u * scratch[2 * a]);
    Uci[t] = (float)((double)u * scratch[2 * a + 1]);
  }
}

// U [dim, r] -> Ut [r, dim], Uc, Uci from imported coefficients.
__global__ void import_layouts_kernel(const float *Uin, const float *cf, const float *ci,
                                      int64_t dim, int r, float *Ut, float *U, float *Uc,
                                      float *Uci) {
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < dim * r;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = t / r;
    const int a = (int)(t % r);
    const float u = Uin[t];
    U[t] = u;
    Ut[(int64_t)a * dim + i] = u;
    Uc[t] = u * cf[a];
    Uci[t] = u * ci[a];
  }
}

__global__ void fill_f32_kernel(float *p, int64_t n, float v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

unsigned grid_for(int64_t n, int64_t per = 256, int64_t cap = 8192) {
  int64_t g = (n + per - 1) / per;
  if (g < 1) g = 1;
  return (unsigned)(g > cap ? cap : g);
}

size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

}  // namespace

gift_status side_set_identity(gift_ctx *ctx, Side &s) {
  const int64_t nr = s.dim * s.r;
  hipLaunchKernelGGL(fill_f32_kernel, dim3(grid_for(nr)), dim3(256), 0, ctx->stream, s.U, nr, 0.f);
  hipLaunchKernelGGL(fill_f32_kernel, dim3(grid_for(nr)), dim3(256), 0, ctx->stream, s.Ut, nr, 0.f);
  hipLaunchKernelGGL(fill_f32_kernel, dim3(grid_for(nr)), dim3(256), 0, ctx->stream, s.Uc, nr, 0.f);
  hipLaunchKernelGGL(fill_f32_kernel, dim3(grid_for(nr)), dim3(256), 0, ctx->stream, s.Uci, nr, 0.f);
  hipLaunchKernelGGL(fill_f32_kernel, dim3(1), dim3(256), 0, ctx->stream, s.c_fwd, (int64_t)s.r, 0.f);
  hipLaunchKernelGGL(fill_f32_kernel, dim3(1), dim3(256), 0, ctx->stream, s.c_inv, (int64_t)s.r, 0.f);
  hipLaunchKernelGGL(fill_f32_kernel, dim3(1), dim3(256), 0, ctx->stream, s.lam, (int64_t)s.r, 0.f);
  hipLaunchKernelGGL(fill_f32_kernel, dim3(1), dim3(64), 0, ctx->stream, s.sigma2, (int64_t)1, 0.f);
  s.have_basis = false;
  return check_launch("side_set_identity");
}

gift_status side_import(gift_ctx *ctx, Side &s, const float *U, const float *c_fwd,
                        const float *c_inv, const float *sigma2) {
  if (s.r == 0) return GIFT_OK;
  GIFT_HIP_TRY(hipMemcpyAsync(s.c_fwd, c_fwd, sizeof(float) * s.r, hipMemcpyDeviceToDevice, ctx->stream));
  GIFT_HIP_TRY(hipMemcpyAsync(s.c_inv, c_inv, sizeof(float) * s.r, hipMemcpyDeviceToDevice, ctx->stream));
  GIFT_HIP_TRY(hipMemcpyAsync(s.sigma2, sigma2, sizeof(float), hipMemcpyDeviceToDevice, ctx->stream));
  hipLaunchKernelGGL(import_layouts_kernel, dim3(grid_for(s.dim * s.r)), dim3(256), 0, ctx->stream,
                     U, c_fwd, c_inv, s.dim, s.r, s.Ut, s.U, s.Uc, s.Uci);
  // warm start of the next refresh: U's rows, then fresh start-block rows
  GIFT_HIP_TRY(hipMemcpyAsync(s.Qt, s.Ut, sizeof(float) * s.dim * s.r, hipMemcpyDeviceToDevice,
                              ctx->stream));
  s.have_basis = true;
  s.fill_tail = true;
  return check_launch("side_import");
}

gift_status side_export(gift_ctx *ctx, const Side &s, float *U, float *c_fwd, float *c_inv,
                        float *sigma2) {
  if (s.r > 0) {
    GIFT_HIP_TRY(hipMemcpyAsync(U, s.U, sizeof(float) * s.dim * s.r, hipMemcpyDeviceToDevice, ctx->stream));
    GIFT_HIP_TRY(hipMemcpyAsync(c_fwd, s.c_fwd, sizeof(float) * s.r, hipMemcpyDeviceToDevice, ctx->stream));
    GIFT_HIP_TRY(hipMemcpyAsync(c_inv, s.c_inv, sizeof(float) * s.r, hipMemcpyDeviceToDevice, ctx->stream));
  }
  GIFT_HIP_TRY(hipMemcpyAsync(sigma2, s.sigma2, sizeof(float), hipMemcpyDeviceToDevice, ctx->stream));
  return GIFT_OK;
}

// One side's refresh.  x: [T, dim] activations (input side) or output
// gradients (output side).
gift_status factor_refresh_side(gift_ctx *ctx, gift_factor *f, Side &s, const void *x,
                                int64_t T, gift_dtype dtype, int32_t iters, uint64_t seed) {
  if (s.r == 0) return GIFT_OK;
  const int64_t dim = s.dim;
  const int k = s.k, r = s.r;
  const int ks = (int)((dim + 255) / 256);  // split-K factor of the k x k products
  // workspace carve-up
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align256(bytes);
    return o;
  };
  const size_t o_A = take(sizeof(float) * dim * dim);
  const size_t o_X = dtype == GIFT_BF16 ? take(sizeof(float) * T * dim) : 0;
  const size_t o_Y = take(sizeof(float) * (size_t)k * dim);
  const size_t o_P = take(sizeof(float) * (size_t)ks * k * k);
  const size_t o_R = take(sizeof(float) * (size_t)k * k);
  const size_t o_W = take(sizeof(double) * (size_t)k * k);
  const size_t o_X2 = take(sizeof(double) * (size_t)k * k);
  const size_t o_th = take(sizeof(double) * (size_t)k);
  const size_t o_nm = take(sizeof(double) * (size_t)k);
  const size_t o_V = take(sizeof(float) * (size_t)k * r);
  const size_t o_sc = take(sizeof(double) * 2 * (size_t)r);
  void *base = nullptr;
  gift_status st = workspace(ctx, off, &base);
  if (st != GIFT_OK) return st;
  char *b = static_cast<char *>(base);
  float *Amat = reinterpret_cast<float *>(b + o_A);
  float *Y = reinterpret_cast<float *>(b + o_Y);
  float *part = reinterpret_cast<float *>(b + o_P);
  float *Rinv = reinterpret_cast<float *>(b + o_R);
  double *W = reinterpret_cast<double *>(b + o_W);
  double *X2 = reinterpret_cast<double *>(b + o_X2);
  double *theta = reinterpret_cast<double *>(b + o_th);
  double *norms = reinterpret_cast<double *>(b + o_nm);
  float *Vr = reinterpret_cast<float *>(b + o_V);
  double *sc = reinterpret_cast<double *>(b + o_sc);
  hipStream_t stream = ctx->stream;

  // 1. statistics A = X^T X / T
  const float *X32 = static_cast<const float *>(x);
  if (dtype == GIFT_BF16) {
    float *Xc = reinterpret_cast<float *>(b + o_X);
    {
      ProfileScope prof(ctx, GIFT_KERNEL_SYRK);
      hipLaunchKernelGGL(bf16_to_f32_kernel, dim3(grid_for(T * dim)), dim3(256), 0, stream, Xc,
                         static_cast<const uint16_t *>(x), T * dim);
    }
    if ((st = check_launch("bf16_to_f32_kernel")) != GIFT_OK) return st;
    X32 = Xc;
  }
  {
    TileJob j;
    j.nseg = 1;
    j.seg[0].a = Operand{X32, dim, 0, false};   // (i, t) = X[t][i]
    j.seg[0].b = Operand{X32, dim, 0, false};   // (t, j) = X[t][j]
    j.seg[0].K = T;
    j.M = dim;
    j.N = dim;
    j.C = Amat;
    j.ldc = dim;
    j.alpha = (float)(1.0 / (double)T);
    j.kernel_family = GIFT_KERNEL_SYRK;
    if ((st = launch_tile(ctx, j)) != GIFT_OK) return st;
  }

  // 2. start block (cold), or the imported basis completed with start rows
  if (!s.have_basis || s.fill_tail) {
    const int row0 = s.have_basis ? r : 0;
    if (row0 < k) {
      ProfileScope prof(ctx, GIFT_KERNEL_FACTOR);
      hipLaunchKernelGGL(start_block_kernel, dim3(grid_for((int64_t)(k - row0) * dim)), dim3(256),
                         0, stream, s.Qt, dim, k, row0, (uint32_t)(seed & 0xffffffffu),
                         (uint32_t)(seed >> 32));
    }
    if ((st = check_launch("start_block_kernel")) != GIFT_OK) return st;
    s.fill_tail = false;
  }

  // Gram / projected-matrix partials: part[z] = Lt_z Rt_z^T over K slice z
  auto kk_product = [&](const float *Lt, const float *Rt) -> gift_status {
    TileJob j;
    j.nseg = 1;
    j.seg[0].a = Operand{Lt, dim, 0, true};
    j.seg[0].b = Operand{Rt, dim, 0, true};
    j.seg[0].K = dim;
    j.M = k;
    j.N = k;
    j.ksplit = ks;
    j.C = part;
    j.ldc = k;
    j.cbs = (int64_t)k * k;
    j.kernel_family = GIFT_KERNEL_FACTOR;
    return launch_tile(ctx, j);
  };
  // Qt <- Rinv^T Src  (Q = Y R^-1)
  auto apply_rinv = [&](const float *Src) -> gift_status {
    TileJob j;
    j.nseg = 1;
    j.seg[0].a = Operand{Rinv, k, 0, false};   // (a, c) = Rinv[c][a]
    j.seg[0].b = Operand{Src, dim, 0, false};  // (c, i) = Src[c][i]
    j.seg[0].K = k;
    j.M = k;
    j.N = dim;
    j.C = s.Qt;
    j.ldc = dim;
    j.kernel_family = GIFT_KERNEL_FACTOR;
    return launch_tile(ctx, j);
  };
  auto cholqr_pass = [&](const float *Src) -> gift_status {
    gift_status e = kk_product(Src, Src);
    if (e != GIFT_OK) return e;
    {
      ProfileScope prof(ctx, GIFT_KERNEL_FACTOR);
      hipLaunchKernelGGL(chol_inv_kernel, dim3(1), dim3(kSmallThreads), 0, stream, part, ks, k, W,
                         X2, Rinv);
    }
    if ((e = check_launch("chol_inv_kernel")) != GIFT_OK) return e;
    return apply_rinv(Src);
  };
  // Yt = Qt A (A symmetric, so (c, i) = A[i][c] reads K-major)
  auto times_A = [&]() -> gift_status {
    TileJob j;
    j.nseg = 1;
    j.seg[0].a = Operand{s.Qt, dim, 0, true};
    j.seg[0].b = Operand{Amat, dim, 0, true};
    j.seg[0].K = dim;
    j.M = k;
    j.N = dim;
    j.C = Y;
    j.ldc = dim;
    j.kernel_family = GIFT_KERNEL_FACTOR;
    return launch_tile(ctx, j);
  };

  // CholQR2 of Y into Qt: two passes, each reading Y and writing Qt
  auto cholqr2 = [&]() -> gift_status {
    gift_status e = cholqr_pass(Y);
    if (e != GIFT_OK) return e;
    GIFT_HIP_TRY(hipMemcpyAsync(Y, s.Qt, sizeof(float) * k * dim, hipMemcpyDeviceToDevice, stream));
    return cholqr_pass(Y);
  };
  GIFT_HIP_TRY(hipMemcpyAsync(Y, s.Qt, sizeof(float) * k * dim, hipMemcpyDeviceToDevice, stream));
  if ((st = cholqr2()) != GIFT_OK) return st;
  for (int it = 0; it < iters; ++it) {
    if ((st = times_A()) != GIFT_OK) return st;
    if ((st = cholqr2()) != GIFT_OK) return st;
  }
  // Rayleigh-Ritz
  if ((st = times_A()) != GIFT_OK) return st;
  if ((st = kk_product(s.Qt, Y)) != GIFT_OK) return st;
  {
    ProfileScope prof(ctx, GIFT_KERNEL_FACTOR);
    hipLaunchKernelGGL(rr_eig_kernel, dim3(1), dim3(kSmallThreads), 0, stream, part, ks, k, r, W,
                       norms, theta, Vr, 30);
  }
  if ((st = check_launch("rr_eig_kernel")) != GIFT_OK) return st;
  {
    TileJob j;  // Ut = Vr^T Qt
    j.nseg = 1;
    j.seg[0].a = Operand{Vr, r, 0, false};     // (a, c) = Vr[c][a]
    j.seg[0].b = Operand{s.Qt, dim, 0, false}; // (c, i) = Qt[c][i]
    j.seg[0].K = k;
    j.M = r;
    j.N = dim;
    j.C = s.Ut;
    j.ldc = dim;
    j.kernel_family = GIFT_KERNEL_FACTOR;
    if ((st = launch_tile(ctx, j)) != GIFT_OK) return st;
  }
  {
    ProfileScope prof(ctx, GIFT_KERNEL_FACTOR);
    hipLaunchKernelGGL(finalize_kernel, dim3(1), dim3(kSmallThreads), 0, stream, Amat, dim, theta, r,
                       f->damping, s.Ut, s.U, s.Uc, s.Uci, s.c_fwd, s.c_inv, s.lam, s.sigma2, sc);
  }
  if ((st = check_launch("finalize_kernel")) != GIFT_OK) return st;
  s.have_basis = true;
  return GIFT_OK;
}

}  // namespace gift
