// Factor refresh: K-FAC statistics and their rank-r transform, batched over
// all factor sides of one dimension.
//
// A = X^T X / T (eq. kfac_fisher_block, eq. impl_A_psd), then its leading r
// eigenpairs (eq. impl_A_lowrank) by block subspace iteration with
// k = min(dim, 2r) columns:
//
//   Q <- CholQR2(start);  repeat iters: Q <- CholQR2(A Q)
//   B = Q^T A Q;  B = V diag(theta) V^T (theta descending);  U = Q V[:, :r]
//
// (Golub & Van Loan, Matrix Computations, Sec. 8.2.4 and 8.1.6; CholeskyQR2
// after Fukaya et al. 2014.)  The dense products run on the tile kernel's FP32
// MFMA path with the members of a batch as its batch dimension.  The k x k
// steps (Cholesky with its triangular inverse, the symmetric eigensolver) are
// single-workgroup kernels in float64, one workgroup per member, working in
// LDS when k <= 128.  The eigensolver is one-sided (Hestenes) Jacobi with
// round-robin parallel ordering: rotating the columns of the symmetric
// positive semidefinite B until they are mutually orthogonal yields
// B V = V diag(theta), so column norms are the eigenvalues and normalised
// columns the eigenvectors.
//
// The next refresh warm-starts from the rotated basis Q V (all k columns,
// descending Ritz values), which leaves B nearly diagonal after one more
// iteration, so the eigensolver then needs few sweeps.
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

#include <algorithm>
#include <map>
#include <vector>

#include "gift_internal.h"

namespace gift {

gift_status launch_syrk_bf16(gift_ctx *ctx, const uint16_t *const *x_table, int members,
                             int64_t T, int64_t dim, float scale, float *A);

namespace {

constexpr int kSmallThreads = 1024;
constexpr int kLdsK = 128;   // k handled in LDS by the small kernels
// Columns count as orthogonal once |<p,q>| <= 1e-10 |p| |q|: B comes from
// float32 products (relative noise ~1e-7), so rotating further changes nothing
// the codec can see.
constexpr double kJacobiTol = 1e-10;

// Per-member state pointers, read by the gather / scatter kernels.
struct Member {
  float *Qt, *Ut, *U, *Uc, *Uci, *c_fwd, *c_inv, *lam, *sigma2;
  uint32_t seed_lo, seed_hi;
  int mode;        // 0 cold start, 1 warm start, 2 imported U + start rows
  float damping;
};

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

// Qw[member] (k x dim, rows = basis vectors): warm rows from the member's
// Qt, the others from the start block.
__global__ void gather_start_kernel(const Member *mem, float *Qw, int64_t dim, int k, int r) {
  const int g = blockIdx.y;
  const Member M = mem[g];
  const int64_t total = (int64_t)k * dim;
  float *dst = Qw + (int64_t)g * total;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int j = (int)(t / dim);
    const int64_t i = t % dim;
    const bool warm = M.mode == 1 || (M.mode == 2 && j < r);
    float v;
    if (warm) {
      v = M.Qt[t];
    } else {
      const uint32_t w = philox_word0((uint32_t)i, (uint32_t)j, 0u, 0u, M.seed_lo, M.seed_hi);
      v = (float)(((int32_t)w) >> 8) * 1.1920928955078125e-7f;
    }
    dst[t] = v;
  }
}

__global__ void bf16_to_f32_kernel(float *dst, const uint16_t *src, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = __uint_as_float((uint32_t)src[i] << 16);
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

// ---------------------------------------------------------------------------
// Cholesky of the Gram matrix and its triangular inverse.
// W (k x k, float64) is LDS or global scratch.  R (upper, pivots floored at
// 1e-12 tr/k) replaces the upper triangle; X = R^-1 is kept transposed in the
// strict lower triangle with its diagonal in xdiag.  Output Rinv (float32).
// ---------------------------------------------------------------------------
__device__ void chol_inv_body(const float *part, int ks, int k, double *W, double *xdiag,
                              double *red, float *Rinv) {
  const int tid = threadIdx.x, nt = blockDim.x;
  const int64_t kk = (int64_t)k * k;
  for (int64_t t = tid; t < kk; t += nt) {
    double s = 0.0;
    for (int z = 0; z < ks; ++z) s += (double)part[z * kk + t];
    W[t] = s;
  }
  __syncthreads();
  double tr = 0.0;
  for (int i = tid; i < k; i += nt) tr += W[(int64_t)i * k + i];
  tr = block_sum(tr, red);
  const double floor = 1e-12 * (tr > 0.0 ? tr : 0.0) / (k > 0 ? k : 1) + 1e-300;
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
  // X = R^-1, bottom row first; 8 lanes per column share each dot product
  for (int i = k - 1; i >= 0; --i) {
    const double rii = W[(int64_t)i * k + i];
    for (int base = 0; base < k; base += nt / 8) {
      const int c = i + 1 + base + tid / 8, part8 = tid & 7;
      double s = 0.0;
      if (c < k) {
        for (int l = i + 1 + part8; l <= c; l += 8)
          s += W[(int64_t)i * k + l] * (l == c ? xdiag[c] : W[(int64_t)c * k + l]);
      }
      s += __shfl_xor(s, 1);
      s += __shfl_xor(s, 2);
      s += __shfl_xor(s, 4);
      if (c < k && part8 == 0) W[(int64_t)c * k + i] = -s / rii;
    }
    if (tid == 0) xdiag[i] = 1.0 / rii;
    __syncthreads();
  }
  for (int64_t t = tid; t < kk; t += nt) {
    const int i = (int)(t / k), c = (int)(t % k);
    double v = 0.0;
    if (c > i) v = W[(int64_t)c * k + i];
    else if (c == i) v = xdiag[i];
    Rinv[t] = (float)v;
  }
}

__global__ __launch_bounds__(kSmallThreads) void chol_inv_lds_kernel(const float *part, int ks, int k,
                                                                     float *Rinv) {
  __shared__ double W[kLdsK * kLdsK];
  __shared__ double xdiag[kLdsK];
  __shared__ double red[kSmallThreads];
  const int g = blockIdx.x;
  chol_inv_body(part + (int64_t)g * ks * k * k, ks, k, W, xdiag, red, Rinv + (int64_t)g * k * k);
}

__global__ __launch_bounds__(kSmallThreads) void chol_inv_global_kernel(const float *part, int ks,
                                                                        int k, double *Wg,
                                                                        double *xdg, float *Rinv) {
  __shared__ double red[kSmallThreads];
  const int g = blockIdx.x;
  chol_inv_body(part + (int64_t)g * ks * k * k, ks, k, Wg + (int64_t)g * k * k, xdg + (int64_t)g * k,
                red, Rinv + (int64_t)g * k * k);
}

// ---------------------------------------------------------------------------
// Rayleigh-Ritz eigensolver: B (partials, symmetrised) -> V (k x k, columns
// sorted by descending eigenvalue) and theta (k).  One-sided Jacobi on the
// columns of W (column-major, W[c*k + row]); 16 lanes per column pair.
// ---------------------------------------------------------------------------
__device__ void rr_eig_body(const float *part, int ks, int k, double *W, double *norms,
                            int *any_rot, float *V, float *theta, int max_sweeps) {
  const int tid = threadIdx.x, nt = blockDim.x;
  const int64_t kk = (int64_t)k * k;
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
  const int kp = (k + 1) & ~1;
  const int npairs = kp / 2;
  const int lanes = 16;
  const int groups = nt / lanes;
  for (int sweep = 0; sweep < max_sweeps; ++sweep) {
    if (tid == 0) *any_rot = 0;
    __syncthreads();
    for (int round = 0; round < kp - 1; ++round) {
      for (int pb = 0; pb < npairs; pb += groups) {
        const int pi = pb + tid / lanes, part16 = tid % lanes;
        int p = 0, q = 0;
        bool valid = pi < npairs;
        if (valid) {
          if (pi == 0) {
            p = round;
            q = kp - 1;
          } else {
            p = (round + pi) % (kp - 1);
            q = (round - pi + kp - 1) % (kp - 1);
          }
          if (p > q) {
            const int tt = p;
            p = q;
            q = tt;
          }
          valid = q < k;
        }
        double alpha = 0.0, beta = 0.0, gamma = 0.0;
        if (valid) {
          const double *cp = W + (int64_t)p * k, *cq = W + (int64_t)q * k;
          for (int i = part16; i < k; i += lanes) {
            const double a = cp[i], b = cq[i];
            alpha += a * a;
            beta += b * b;
            gamma += a * b;
          }
        }
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) {
          alpha += __shfl_xor(alpha, o);
          beta += __shfl_xor(beta, o);
          gamma += __shfl_xor(gamma, o);
        }
        if (valid && gamma != 0.0 && fabs(gamma) > kJacobiTol * sqrt(alpha * beta)) {
          const double zeta = (beta - alpha) / (2.0 * gamma);
          const double t = (zeta >= 0.0 ? 1.0 : -1.0) / (fabs(zeta) + sqrt(1.0 + zeta * zeta));
          const double c = 1.0 / sqrt(1.0 + t * t);
          const double s = c * t;
          double *cp = W + (int64_t)p * k, *cq = W + (int64_t)q * k;
          for (int i = part16; i < k; i += lanes) {
            const double a = cp[i], b = cq[i];
            cp[i] = c * a - s * b;
            cq[i] = s * a + c * b;
          }
          if (part16 == 0) *any_rot = 1;
        }
        if (npairs > groups) __syncthreads();
      }
      __syncthreads();
    }
    const int rotated = *any_rot;
    __syncthreads();
    if (!rotated) break;
  }
  for (int j = tid; j < k; j += nt) {
    double s = 0.0;
    for (int i = 0; i < k; ++i) s += W[(int64_t)j * k + i] * W[(int64_t)j * k + i];
    norms[j] = sqrt(s);
  }
  __syncthreads();
  for (int j = tid; j < k; j += nt) {
    const double v = norms[j];
    int rank = 0;
    for (int l = 0; l < k; ++l) {
      const double u = norms[l];
      rank += (u > v) || (u == v && l < j);
    }
    theta[rank] = (float)v;
    const double inv = v > 0.0 ? 1.0 / v : 0.0;
    for (int i = 0; i < k; ++i) V[(int64_t)i * k + rank] = (float)(W[(int64_t)j * k + i] * inv);
  }
}

__global__ __launch_bounds__(kSmallThreads) void rr_eig_lds_kernel(const float *part, int ks, int k,
                                                                   float *V, float *theta,
                                                                   int max_sweeps) {
  __shared__ double W[kLdsK * kLdsK];
  __shared__ double norms[kLdsK];
  __shared__ int any_rot;
  const int g = blockIdx.x;
  rr_eig_body(part + (int64_t)g * ks * k * k, ks, k, W, norms, &any_rot, V + (int64_t)g * k * k,
              theta + (int64_t)g * k, max_sweeps);
}

__global__ __launch_bounds__(kSmallThreads) void rr_eig_global_kernel(const float *part, int ks,
                                                                      int k, double *Wg,
                                                                      double *ng, float *V,
                                                                      float *theta,
                                                                      int max_sweeps) {
  __shared__ int any_rot;
  const int g = blockIdx.x;
  rr_eig_body(part + (int64_t)g * ks * k * k, ks, k, Wg + (int64_t)g * k * k, ng + (int64_t)g * k,
              &any_rot, V + (int64_t)g * k * k, theta + (int64_t)g * k, max_sweeps);
}

// sigma^2, coefficients, U layouts and the warm-start block of each member.
__global__ __launch_bounds__(kSmallThreads) void finalize_kernel(const Member *mem,
                                                                 const float *Amat, int64_t dim,
                                                                 const float *theta, int k, int r,
                                                                 const float *Qrot) {
  __shared__ double red[kSmallThreads];
  __shared__ double coef[2 * 512];
  const int g = blockIdx.x;
  const Member M = mem[g];
  const float *A = Amat + (int64_t)g * dim * dim;
  const float *th = theta + (int64_t)g * k;
  const float *Q = Qrot + (int64_t)g * k * dim;
  const int tid = threadIdx.x, nt = blockDim.x;
  double tr = 0.0;
  for (int64_t i = tid; i < dim; i += nt) tr += (double)A[i * dim + i];
  tr = block_sum(tr, red);
  double top = 0.0;
  for (int i = tid; i < r; i += nt) top += th[i] > 0.f ? (double)th[i] : 0.0;
  top = block_sum(top, red);
  const bool identity = !(tr > 0.0) || r == 0;
  const double floor = (double)M.damping * tr / (double)dim;
  double sigma2 = 0.0;
  if (!identity) {
    if (r >= dim) {
      sigma2 = tr / (double)dim;
    } else {
      sigma2 = (tr - top) / (double)(dim - r);
      if (sigma2 < floor) sigma2 = floor;
    }
  }
  for (int i = tid; i < r; i += nt) {
    double l = th[i] > 0.f ? (double)th[i] : 0.0;
    double cf = 0.0, ci = 0.0;
    if (!identity) {
      const double fl = r >= dim ? floor : sigma2;
      if (l < fl) l = fl;
      cf = sqrt(sigma2 / l) - 1.0;
      ci = sqrt(l / sigma2) - 1.0;
    }
    coef[2 * i] = cf;
    coef[2 * i + 1] = ci;
    M.c_fwd[i] = (float)cf;
    M.c_inv[i] = (float)ci;
    M.lam[i] = (float)l;
  }
  if (tid == 0) M.sigma2[0] = (float)sigma2;
  __syncthreads();
  for (int64_t t = tid; t < (int64_t)k * dim; t += nt) M.Qt[t] = Q[t];
  for (int64_t t = tid; t < (int64_t)r * dim; t += nt) M.Ut[t] = Q[t];
  for (int64_t t = tid; t < dim * r; t += nt) {
    const int64_t i = t / r;
    const int a = (int)(t % r);
    const float u = Q[(int64_t)a * dim + i];
    M.U[t] = u;
    M.Uc[t] = (float)((double)u * coef[2 * a]);
    M.Uci[t] = (float)((double)u * coef[2 * a + 1]);
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
  float *bufs[4] = {s.U, s.Ut, s.Uc, s.Uci};
  for (float *b : bufs)
    hipLaunchKernelGGL(fill_f32_kernel, dim3(grid_for(nr)), dim3(256), 0, ctx->stream, b, nr, 0.f);
  float *small[3] = {s.c_fwd, s.c_inv, s.lam};
  for (float *b : small)
    hipLaunchKernelGGL(fill_f32_kernel, dim3(1), dim3(256), 0, ctx->stream, b, (int64_t)s.r, 0.f);
  hipLaunchKernelGGL(fill_f32_kernel, dim3(1), dim3(64), 0, ctx->stream, s.sigma2, (int64_t)1, 0.f);
  s.have_basis = false;
  s.fill_tail = false;
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
  // warm start of the next refresh: U's rows, then start-block rows
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

// Refresh a group of sides with equal (dim, r): one launch sequence for all.
static gift_status refresh_group(gift_ctx *ctx, const std::vector<SideJob> &jobs, int64_t T,
                                 gift_dtype dtype, int32_t iters) {
  const int G = (int)jobs.size();
  const Side &s0 = *jobs[0].side;
  const int64_t dim = s0.dim;
  const int k = s0.k, r = s0.r;
  const int ks = (int)((dim + 255) / 256);   // split-K factor of the k x k products
  const bool lds = k <= kLdsK;
  const bool bf16_direct = dtype == GIFT_BF16 && dim % 8 == 0;
  // workspace carve-up
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align256(bytes);
    return o;
  };
  const size_t o_tab = take(sizeof(Member) * G);
  const size_t o_xt = take(sizeof(void *) * G);
  const size_t o_A = take(sizeof(float) * G * dim * dim);
  const size_t o_X = (dtype == GIFT_BF16 && !bf16_direct) ? take(sizeof(float) * T * dim) : 0;
  const size_t o_Q = take(sizeof(float) * G * (size_t)k * dim);
  const size_t o_Y = take(sizeof(float) * G * (size_t)k * dim);
  const size_t o_P = take(sizeof(float) * G * (size_t)ks * k * k);
  const size_t o_R = take(sizeof(float) * G * (size_t)k * k);
  const size_t o_V = take(sizeof(float) * G * (size_t)k * k);
  const size_t o_th = take(sizeof(float) * G * (size_t)k);
  const size_t o_W = lds ? 0 : take(sizeof(double) * G * (size_t)k * k);
  const size_t o_x2 = lds ? 0 : take(sizeof(double) * G * (size_t)k);
  void *base = nullptr;
  gift_status st = workspace(ctx, off, &base);
  if (st != GIFT_OK) return st;
  char *b = static_cast<char *>(base);
  Member *tab = reinterpret_cast<Member *>(b + o_tab);
  const void **xtab = reinterpret_cast<const void **>(b + o_xt);
  float *Amat = reinterpret_cast<float *>(b + o_A);
  float *Qw = reinterpret_cast<float *>(b + o_Q);
  float *Y = reinterpret_cast<float *>(b + o_Y);
  float *part = reinterpret_cast<float *>(b + o_P);
  float *Rinv = reinterpret_cast<float *>(b + o_R);
  float *V = reinterpret_cast<float *>(b + o_V);
  float *theta = reinterpret_cast<float *>(b + o_th);
  double *Wg = lds ? nullptr : reinterpret_cast<double *>(b + o_W);
  double *x2 = lds ? nullptr : reinterpret_cast<double *>(b + o_x2);
  hipStream_t stream = ctx->stream;

  // member table (copied from pageable host memory: staged before returning)
  std::vector<Member> host(G);
  std::vector<const void *> xs(G);
  bool any_cold = false;
  for (int g = 0; g < G; ++g) {
    const Side &s = *jobs[g].side;
    Member &M = host[g];
    M.Qt = s.Qt;
    M.Ut = s.Ut;
    M.U = s.U;
    M.Uc = s.Uc;
    M.Uci = s.Uci;
    M.c_fwd = s.c_fwd;
    M.c_inv = s.c_inv;
    M.lam = s.lam;
    M.sigma2 = s.sigma2;
    M.seed_lo = (uint32_t)(jobs[g].seed & 0xffffffffu);
    M.seed_hi = (uint32_t)(jobs[g].seed >> 32);
    M.mode = !s.have_basis ? 0 : (s.fill_tail ? 2 : 1);
    M.damping = jobs[g].damping;
    any_cold = any_cold || M.mode != 1;
    xs[g] = jobs[g].x;
  }
  GIFT_HIP_TRY(hipMemcpyAsync(tab, host.data(), sizeof(Member) * G, hipMemcpyHostToDevice, stream));
  GIFT_HIP_TRY(hipMemcpyAsync(xtab, xs.data(), sizeof(void *) * G, hipMemcpyHostToDevice, stream));

  // 1. statistics A_g = X_g^T X_g / T
  const float inv_T = (float)(1.0 / (double)T);
  if (bf16_direct) {
    if ((st = launch_syrk_bf16(ctx, reinterpret_cast<const uint16_t *const *>(xtab), G, T, dim,
                               inv_T, Amat)) != GIFT_OK)
      return st;
  } else {
    for (int g = 0; g < G; ++g) {
      const float *X32 = static_cast<const float *>(jobs[g].x);
      if (dtype == GIFT_BF16) {
        float *Xc = reinterpret_cast<float *>(b + o_X);
        {
          ProfileScope prof(ctx, GIFT_KERNEL_SYRK);
          hipLaunchKernelGGL(bf16_to_f32_kernel, dim3(grid_for(T * dim)), dim3(256), 0, stream, Xc,
                             static_cast<const uint16_t *>(jobs[g].x), T * dim);
        }
        if ((st = check_launch("bf16_to_f32_kernel")) != GIFT_OK) return st;
        X32 = Xc;
      }
      TileJob j;
      j.nseg = 1;
      j.seg[0].a = Operand{X32, dim, 0, false};   // (i, t) = X[t][i]
      j.seg[0].b = Operand{X32, dim, 0, false};   // (t, j) = X[t][j]
      j.seg[0].K = T;
      j.M = dim;
      j.N = dim;
      j.C = Amat + (int64_t)g * dim * dim;
      j.ldc = dim;
      j.alpha = inv_T;
      j.kernel_family = GIFT_KERNEL_SYRK;
      if ((st = launch_tile(ctx, j)) != GIFT_OK) return st;
    }
  }

  // 2. start blocks
  {
    ProfileScope prof(ctx, GIFT_KERNEL_FACTOR);
    hipLaunchKernelGGL(gather_start_kernel, dim3(grid_for((int64_t)k * dim, 256, 2048), G), dim3(256),
                       0, stream, tab, Qw, dim, k, r);
  }
  if ((st = check_launch("gather_start_kernel")) != GIFT_OK) return st;

  const int64_t kd = (int64_t)k * dim, k2 = (int64_t)k * k;
  // part[g][z] = Lt_g Rt_g^T over K slice z
  auto kk_product = [&](const float *Lt, const float *Rt) -> gift_status {
    TileJob j;
    j.nseg = 1;
    j.seg[0].a = Operand{Lt, dim, kd, true};
    j.seg[0].b = Operand{Rt, dim, kd, true};
    j.seg[0].K = dim;
    j.M = k;
    j.N = k;
    j.batch = G;
    j.ksplit = ks;
    j.C = part;
    j.ldc = k;
    j.cbs = k2;
    j.kernel_family = GIFT_KERNEL_FACTOR;
    return launch_tile(ctx, j);
  };
  // Qw <- Rinv^T Y  (Q = Y R^-1)
  auto apply_rinv = [&]() -> gift_status {
    TileJob j;
    j.nseg = 1;
    j.seg[0].a = Operand{Rinv, k, k2, false};   // (a, c) = Rinv[c][a]
    j.seg[0].b = Operand{Y, dim, kd, false};    // (c, i) = Y[c][i]
    j.seg[0].K = k;
    j.M = k;
    j.N = dim;
    j.batch = G;
    j.C = Qw;
    j.ldc = dim;
    j.cbs = kd;
    j.kernel_family = GIFT_KERNEL_FACTOR;
    return launch_tile(ctx, j);
  };
  auto cholqr_pass = [&]() -> gift_status {
    gift_status e = kk_product(Y, Y);
    if (e != GIFT_OK) return e;
    {
      ProfileScope prof(ctx, GIFT_KERNEL_FACTOR);
      if (lds)
        hipLaunchKernelGGL(chol_inv_lds_kernel, dim3(G), dim3(kSmallThreads), 0, stream, part, ks, k, Rinv);
      else
        hipLaunchKernelGGL(chol_inv_global_kernel, dim3(G), dim3(kSmallThreads), 0, stream, part, ks, k,
                           Wg, x2, Rinv);
    }
    if ((e = check_launch("chol_inv_kernel")) != GIFT_OK) return e;
    return apply_rinv();
  };
  // CholQR2 of Y into Qw
  auto cholqr2 = [&]() -> gift_status {
    gift_status e = cholqr_pass();
    if (e != GIFT_OK) return e;
    GIFT_HIP_TRY(hipMemcpyAsync(Y, Qw, sizeof(float) * G * kd, hipMemcpyDeviceToDevice, stream));
    return cholqr_pass();
  };
  // Y_g = Qw_g A_g  (A symmetric, so (c, i) = A[i][c] reads K-major)
  auto times_A = [&]() -> gift_status {
    TileJob j;
    j.nseg = 1;
    j.seg[0].a = Operand{Qw, dim, kd, true};
    j.seg[0].b = Operand{Amat, dim, dim * dim, true};
    j.seg[0].K = dim;
    j.M = k;
    j.N = dim;
    j.batch = G;
    j.C = Y;
    j.ldc = dim;
    j.cbs = kd;
    j.kernel_family = GIFT_KERNEL_FACTOR;
    return launch_tile(ctx, j);
  };

  if (any_cold) {
    GIFT_HIP_TRY(hipMemcpyAsync(Y, Qw, sizeof(float) * G * kd, hipMemcpyDeviceToDevice, stream));
    if ((st = cholqr2()) != GIFT_OK) return st;
  }
  for (int it = 0; it < iters; ++it) {
    if ((st = times_A()) != GIFT_OK) return st;
    if ((st = cholqr2()) != GIFT_OK) return st;
  }
  // Rayleigh-Ritz: B = Qw A Qw^T, eigenpairs, rotated basis V^T Qw -> Y
  if ((st = times_A()) != GIFT_OK) return st;
  if ((st = kk_product(Qw, Y)) != GIFT_OK) return st;
  {
    ProfileScope prof(ctx, GIFT_KERNEL_FACTOR);
    if (lds)
      hipLaunchKernelGGL(rr_eig_lds_kernel, dim3(G), dim3(kSmallThreads), 0, stream, part, ks, k, V,
                         theta, 40);
    else
      hipLaunchKernelGGL(rr_eig_global_kernel, dim3(G), dim3(kSmallThreads), 0, stream, part, ks, k,
                         Wg, x2, V, theta, 40);
  }
  if ((st = check_launch("rr_eig_kernel")) != GIFT_OK) return st;
  {
    TileJob j;  // Y = V^T Qw
    j.nseg = 1;
    j.seg[0].a = Operand{V, k, k2, false};     // (a, c) = V[c][a]
    j.seg[0].b = Operand{Qw, dim, kd, false};  // (c, i) = Qw[c][i]
    j.seg[0].K = k;
    j.M = k;
    j.N = dim;
    j.batch = G;
    j.C = Y;
    j.ldc = dim;
    j.cbs = kd;
    j.kernel_family = GIFT_KERNEL_FACTOR;
    if ((st = launch_tile(ctx, j)) != GIFT_OK) return st;
  }
  {
    ProfileScope prof(ctx, GIFT_KERNEL_FACTOR);
    hipLaunchKernelGGL(finalize_kernel, dim3(G), dim3(kSmallThreads), 0, stream, tab, Amat, dim, theta,
                       k, r, Y);
  }
  if ((st = check_launch("finalize_kernel")) != GIFT_OK) return st;
  for (const SideJob &jb : jobs) {
    jb.side->have_basis = true;
    jb.side->fill_tail = false;
  }
  return GIFT_OK;
}

gift_status factor_refresh_batch(gift_ctx *ctx, const std::vector<SideJob> &jobs, int64_t T,
                                 gift_dtype dtype, int32_t iters) {
  std::map<std::pair<int64_t, int>, std::vector<SideJob>> groups;
  for (const SideJob &j : jobs)
    if (j.side->r > 0) groups[{j.side->dim, j.side->r}].push_back(j);
  for (auto &kv : groups) {
    gift_status st = refresh_group(ctx, kv.second, T, dtype, iters);
    if (st != GIFT_OK) return st;
  }
  return GIFT_OK;
}

}  // namespace gift
