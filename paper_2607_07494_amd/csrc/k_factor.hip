// Factor refresh: K-FAC statistics and their rank-r transform, batched over
// every factor side of one update call.
//
// A = X^T X / T (eq. kfac_fisher_block, eq. impl_A_psd), then its leading r
// eigenpairs (eq. impl_A_lowrank) by block subspace iteration with
// k = min(dim, 2r) columns:
//
//   Q <- CholQR2(start);  repeat iters: Q <- CholQR2(A Q)
//   B = Q^T A Q;  B = V diag(theta) V^T (theta descending);  U = Q V[:, :r]
//
// (Golub & Van Loan, Matrix Computations, Sec. 8.2.4 and 8.1.6; CholeskyQR2
// after Fukaya et al. 2014.)  Sides are grouped by (dim, r); the dense
// products run once per group on the FP32 MFMA kernels with the group's
// members as the batch dimension, and the groups advance in lockstep so that
// each k x k step is ONE launch over every member of every group: one
// workgroup per member, float64, in LDS when k <= 128.
//
// Cholesky (right-looking, one barrier per column; R^T kept in the strict
// lower triangle) and the inverse of R by forward substitution on R^T, four
// lanes per column.  The eigensolver is one-sided (Hestenes) Jacobi with
// round-robin parallel ordering: rotating the columns of the symmetric
// positive semidefinite B until they are mutually orthogonal yields
// B V = V diag(theta), so column norms are the eigenvalues and normalised
// columns the eigenvectors.  In LDS each column pair is held by 16 lanes in
// registers between its dot products and its rotation, and the dot products
// are reduced with DPP row rotations, which leave bit-identical sums on the
// 16 lanes (every step adds the same two operands on both partner lanes), so
// all lanes of a pair take the same rotation.
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
#include <tuple>
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
constexpr int kEigRegs = 16;   // global eigensolver: a column pair in registers up to k = 256

// One factor side of the refresh.  The side's persistent state, then its
// slices of the group buffers.
struct Member {
  float *Qt, *Ut, *U, *Uc, *Uci, *c_fwd, *c_inv, *lam, *sigma2;
  const float *A;        // statistics [dim, dim]
  float *start;          // start block [k, dim] (rows = basis vectors)
  const float *rot;      // rotated Ritz basis V^T Q [k, dim]
  const float *theta;    // Ritz values [k], descending
  int64_t dim;
  int k, r;
  uint32_t seed_lo, seed_hi;
  int mode;              // 0 cold start, 1 warm start, 2 imported U + start rows
  float damping;
};

// One member's k x k step: partial products in, factor or eigenpairs out.
struct SmallJob {
  const float *part;     // [ks][k][k] split-K partials of the k x k product
  float *out;            // R^-1 (Cholesky) or V (eigensolver), [k][k] row-major
  float *theta;          // eigenvalues [k] (eigensolver)
  double *W;             // [k][k+1] float64 scratch when k > kLdsK
  double *aux;           // [2k + 64] float64 scratch when k > kLdsK
  int ks, k;
  float *rout;           // optional R [k][k] (Cholesky, upper triangular)
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

// start rows of every member: warm rows from the member's Qt, the others from
// the start block (grid.y = member)
__global__ void gather_start_kernel(const Member *mem) {
  const Member M = mem[blockIdx.y];
  const int64_t total = (int64_t)M.k * M.dim;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int j = (int)(t / M.dim);
    const int64_t i = t - (int64_t)j * M.dim;
    const bool warm = M.mode == 1 || (M.mode == 2 && j < M.r);
    float v;
    if (warm) {
      v = M.Qt[t];
    } else {
      const uint32_t w = philox_word0((uint32_t)i, (uint32_t)j, 0u, 0u, M.seed_lo, M.seed_hi);
      v = (float)(((int32_t)w) >> 8) * 1.1920928955078125e-7f;
    }
    M.start[t] = v;
  }
}

__global__ void bf16_to_f32_kernel(float *dst, const uint16_t *src, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = __uint_as_float((uint32_t)src[i] << 16);
}

// v + (v of the lane R places further down the 16-lane DPP row)
template <int R>
__device__ __forceinline__ double ror_add(double v) {
  const int lo = __builtin_amdgcn_mov_dpp(__double2loint(v), 0x120 + R, 0xf, 0xf, false);
  const int hi = __builtin_amdgcn_mov_dpp(__double2hiint(v), 0x120 + R, 0xf, 0xf, false);
  return v + __hiloint2double(hi, lo);
}

// Sum over the 16 lanes of a row; every lane ends with the same bits.
__device__ __forceinline__ double row16_sum(double v) {
  v = ror_add<8>(v);
  v = ror_add<4>(v);
  v = ror_add<2>(v);
  return ror_add<1>(v);
}

// Sum over the 4 lanes of a quad (quad_perm [1,0,3,2] then [2,3,0,1]).
template <int P>
__device__ __forceinline__ double quad_add(double v) {
  const int lo = __builtin_amdgcn_mov_dpp(__double2loint(v), P, 0xf, 0xf, false);
  const int hi = __builtin_amdgcn_mov_dpp(__double2hiint(v), P, 0xf, 0xf, false);
  return v + __hiloint2double(hi, lo);
}
__device__ __forceinline__ double quad_sum(double v) {
  v = quad_add<0xB1>(v);   // quad_perm [1,0,3,2]
  return quad_add<0x4E>(v);  // quad_perm [2,3,0,1]
}
// Sum over the 8 lanes of an octet: quad sums, then row_half_mirror adds the
// other quad's sum (the same two operands on every lane).
__device__ __forceinline__ double octet_sum(double v) {
  return quad_add<0x141>(quad_sum(v));
}

// Sum of the ks split-K partials of a k x k product, element t of [0, kk)
// handed to store(t, value).  Each thread keeps E elements' loads of one
// partial in flight together (a single workgroup reads the whole matrix, so
// the loads must not wait on each other); partials are added in order z = 0..
template <int E, typename F>
__device__ __forceinline__ void sum_partials(const float *part, int ks, int64_t kk, F store) {
  const int tid = threadIdx.x, nt = blockDim.x;
  for (int64_t t0 = 0; t0 < kk; t0 += (int64_t)E * nt) {
    double acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = 0.0;
    for (int z = 0; z < ks; ++z) {
      float v[E];
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int64_t t = t0 + (int64_t)e * nt + tid;
        v[e] = t < kk ? part[z * kk + t] : 0.f;
      }
#pragma unroll
      for (int e = 0; e < E; ++e) acc[e] += (double)v[e];
    }
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int64_t t = t0 + (int64_t)e * nt + tid;
      if (t < kk) store(t, acc[e]);
    }
  }
}

// ---------------------------------------------------------------------------
// Cholesky of the Gram matrix G (sum of the split-K partials) and R^-1.
// W is [k][S] float64 (S = k + 1: rows and columns both hit distinct banks).
// Column j: pivot d = max(G_jj, 1e-12 tr/k), R_jj = sqrt(d),
// R_jl = G_jl / R_jj, trailing G_ab -= R_ja R_jb (upper triangle).  R_jl goes
// to the strict lower triangle W[l][j] (= L = R^T), R_jj to dg[j].  Then
// X = L^-1 column by column (X_cc = 1/L_cc, X_ic = -sum_l L_il X_lc / L_ii),
// X_ic stored at W[c][i]; R^-1 = X^T, row-major float32.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void chol_inv_body(const float *part, int ks, int k, double *W, int S, double *dg,
                                              double *idg, double *sink, float *Rinv, float *Rout) {
  const int tid = threadIdx.x, nt = blockDim.x;
  const int64_t kk = (int64_t)k * k;
  sum_partials<8>(part, ks, kk, [&](int64_t t, double v) {
    const int i = (int)(t / k), j = (int)(t - (int64_t)i * k);
    W[i * S + j] = v;
  });
  __syncthreads();
  double tr = 0.0;   // every thread sums the diagonal in the same order
  for (int i = 0; i < k; ++i) tr += W[i * S + i];
  const double floor = 1e-12 * (tr > 0.0 ? tr : 0.0) / (k > 0 ? k : 1) + 1e-300;
  // trailing update in 4 x 4 register blocks: thread (tx, ty) of a 32 x 32
  // grid takes rows j+1+ty+32u and columns j+1+tx+32v of each 128 x 128 slab
  const int tx = tid & 31, ty = tid >> 5, ty_step = nt >> 5;
  for (int j = 0; j < k; ++j) {
    const double d0 = W[j * S + j];
    const double sj = sqrt(d0 > floor ? d0 : floor);
    const double rs = 1.0 / sj;
    if (tid == 0) dg[j] = sj;
    const int rem = k - j - 1;
    for (int r0 = 0; r0 < rem; r0 += 4 * ty_step) {
      for (int c0 = r0 - r0 % 128; c0 < rem; c0 += 128) {   // column slabs right of the row slab
        // every load is issued unconditionally at a clamped, in-range
        // address (guarded loads would each wait for the one before)
        double ra[4], rb[4], w[4][4];
        int ar[4], bc[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          ar[u] = j + 1 + r0 + ty + ty_step * u;
          bc[u] = j + 1 + c0 + tx + 32 * u;
          const int arc = ar[u] < k ? ar[u] : k - 1, bcc = bc[u] < k ? bc[u] : k - 1;
          ra[u] = W[j * S + arc] * rs;
          rb[u] = W[j * S + bcc] * rs;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int arc = ar[u] < k ? ar[u] : k - 1, bcc = bc[v] < k ? bc[v] : k - 1;
            w[u][v] = W[arc * S + bcc];
          }
        // elements outside the upper trailing triangle go to the sink
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            double *dst = ar[u] <= bc[v] && bc[v] < k ? W + ar[u] * S + bc[v] : sink + (tid & 63);
            *dst = w[u][v] - ra[u] * rb[v];
          }
        if (r0 == 0 && ty == 0) {   // R_jb into the strict lower triangle (column j)
#pragma unroll
          for (int v = 0; v < 4; ++v)
            if (bc[v] < k) W[bc[v] * S + j] = rb[v];
        }
      }
    }
    __syncthreads();
  }
  for (int i = tid; i < k; i += nt) idg[i] = 1.0 / dg[i];
  __syncthreads();
  // X = L^-1: octet o owns column c = o + (nt / 8) u
  const int p = tid & 7;
  for (int c0 = 0; c0 < k; c0 += nt / 8) {
    const int c = c0 + (tid >> 3);
    const bool act = c < k;
    if (act && p == 0) W[c * S + c] = idg[c];
    for (int i = c0 + 1; i < k; ++i) {
      double s = 0.0;
      if (act && c < i) {
        const double *Li = W + i * S, *Xc = W + c * S;
        for (int l0 = c + p; l0 < i; l0 += 32) {
          double lv[4], xv[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int l = l0 + 8 * u < i ? l0 + 8 * u : l0;
            lv[u] = Li[l];
            xv[u] = Xc[l] * (l0 + 8 * u < i ? 1.0 : 0.0);   // finite entries: exact mask
          }
#pragma unroll
          for (int u = 0; u < 4; ++u) s += lv[u] * xv[u];
        }
      }
      s = octet_sum(s);
      if (act && c < i && p == 0) W[c * S + i] = -s * idg[i];
    }
  }
  __syncthreads();
  for (int64_t t = tid; t < kk; t += nt) {
    const int i = (int)(t / k), c = (int)(t - (int64_t)i * k);
    Rinv[t] = c >= i ? (float)W[i * S + c] : 0.f;
  }
  // R: its strict upper part sits transposed in the lower triangle of W
  if (Rout)
    for (int64_t t = tid; t < kk; t += nt) {
      const int i = (int)(t / k), c = (int)(t - (int64_t)i * k);
      Rout[t] = c > i ? (float)W[c * S + i] : (c == i ? (float)dg[i] : 0.f);
    }
}

// ---------------------------------------------------------------------------
// The same factorisation for k <= 128 with the matrices in registers.
// Thread (ty, tx) of a 32 x 32 grid (1024 threads) owns the 4 x 4 block at
// rows 4 ty.., columns 4 tx.. of G when tx >= ty (upper triangle) and of
// X = L^-1 when tx <= ty (lower triangle).  Column step j, with d =
// max(G_jj, floor) and rs = 1 / sqrt(d):
//   the half-wave of block row j / 4 reads G_jj from the lane of the
//   diagonal block, scales its rows j of G and X by rs, keeps the scaled X
//   row (final) and broadcasts both through LDS:
//     l_b = G_jb rs = R_jb = L_bj (b >= j),   x_b = X_jb rs (b <= j);
//   after one barrier every thread updates its blocks with FMAs only:
//     G_ab -= l_a l_b                     (Cholesky trailing update)
//     X_ab -= l_a x_b   for a > j         (Gauss-Jordan on [L | I])
// Two broadcast buffers alternate, so one barrier per column suffices.
// Rows of G at or above j are never read again, so the G update runs over
// whole blocks (stale broadcast entries only reach those rows); the X update
// is restricted to rows below j, whose broadcast entries are current.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kSmallThreads) void chol_inv_lds_kernel(const SmallJob *jobs) {
  __shared__ double lb[2][kLdsK], xb[2][kLdsK];   // broadcast rows of R and X
  __shared__ double dsum[32];
  const SmallJob J = jobs[blockIdx.x];
  const int k = J.k, ks = J.ks;
  const int tid = threadIdx.x, tx = tid & 31, ty = tid >> 5;
  const int64_t kk = (int64_t)k * k;
  const bool own_g = tx >= ty, own_x = tx <= ty;
  double G[4][4], X[4][4];
  // G = sum of the split-K partials (rows / columns past k stay zero)
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      G[u][w] = 0.0;
      X[u][w] = (4 * ty + u == 4 * tx + w && 4 * ty + u < k) ? 1.0 : 0.0;
    }
  if (own_g) {
    for (int z = 0; z < ks; ++z) {
      const float *P = J.part + z * kk;
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const int a = 4 * ty + u, b = 4 * tx + w;
          G[u][w] += (a < k && b < k) ? (double)P[a * k + b] : 0.0;
        }
    }
  }
  // pivot floor from the trace (every thread sums the 32 block sums in order)
  if (tx == ty) dsum[ty] = G[0][0] + G[1][1] + G[2][2] + G[3][3];
  __syncthreads();
  double tr = 0.0;
  for (int i = 0; i < 32; ++i) tr += dsum[i];
  const double floor = 1e-12 * (tr > 0.0 ? tr : 0.0) / (k > 0 ? k : 1) + 1e-300;
  const int half = (tid & 32);   // lane offset of this thread's half-wave

  for (int j = 0; j < k; ++j) {
    const int buf = j & 1, jr = j >> 2, ju = j & 3;
    if (ty == jr) {   // one half-wave: pivot, scaling, broadcast
      double gd = 0.0;
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (u == ju) gd = G[u][u];
      // G_jj from the diagonal block's lane (tx = jr) of this half-wave
      const int src = half + jr;
      const int lo = __builtin_amdgcn_readlane(__double2loint(gd), src);
      const int hi = __builtin_amdgcn_readlane(__double2hiint(gd), src);
      const double d0 = __hiloint2double(hi, lo);
      const double d = d0 > floor ? d0 : floor;
      const double rs = 1.0 / sqrt(d);
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const int col = 4 * tx + w;
        double gv = 0.0, xv = 0.0;
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (u == ju) {
            X[u][w] *= rs;   // row j of X is final from here on
            gv = G[u][w];
            xv = X[u][w];
          }
        const double lv = own_g && col >= j ? gv * rs : 0.0;   // R_j,col
        lb[buf][col] = lv;
        xb[buf][col] = own_x ? xv : 0.0;
        if (J.rout && col < k) J.rout[(int64_t)j * k + col] = (float)lv;
      }
    }
    __syncthreads();
    double la[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) la[u] = lb[buf][4 * ty + u];
    if (own_g && 4 * ty + 3 > j) {
      double lc[4];
#pragma unroll
      for (int w = 0; w < 4; ++w) lc[w] = lb[buf][4 * tx + w];
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int w = 0; w < 4; ++w) G[u][w] -= la[u] * lc[w];
    }
    if (own_x && 4 * ty + 3 > j) {
      double xc[4];
#pragma unroll
      for (int w = 0; w < 4; ++w) xc[w] = xb[buf][4 * tx + w];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (4 * ty + u > j)
#pragma unroll
          for (int w = 0; w < 4; ++w) X[u][w] -= la[u] * xc[w];
    }
  }
  // R^-1 = X^T (upper triangular), row-major: element (i, c) = X[c][i]
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const int c = 4 * ty + u, i = 4 * tx + w;
      if (c < k && i < k) J.out[i * k + c] = own_x ? (float)X[u][w] : 0.f;
    }
}

constexpr int kCholGlobalThreads = 512;   // 64-bit addresses need the register room
__global__ __launch_bounds__(kCholGlobalThreads) void chol_inv_global_kernel(const SmallJob *jobs) {
  const SmallJob J = jobs[blockIdx.x];
  __shared__ double dg[1];  // unused: diagonals live in aux
  (void)dg;
  chol_inv_body(J.part, J.ks, J.k, J.W, J.k + 1, J.aux, J.aux + J.k, J.aux + 2 * J.k, J.out, J.rout);
}

// Givens rotation of the one-sided Jacobi step for columns with squared
// norms alpha, beta and inner product gamma (!= 0).
__device__ __forceinline__ void jacobi_cs(double alpha, double beta, double gamma, double &c,
                                          double &s) {
  const double zeta = (beta - alpha) / (2.0 * gamma);
  const double t = (zeta >= 0.0 ? 1.0 : -1.0) / (fabs(zeta) + sqrt(1.0 + zeta * zeta));
  c = 1.0 / sqrt(1.0 + t * t);
  s = c * t;
}

// round-robin pairing: pair pi of round `round` over kp (even) players
__device__ __forceinline__ void rr_pair(int round, int pi, int kp, int &p, int &q) {
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
}

// B (partials, symmetrised) into column-major W[c*k + row]
template <int E>
__device__ __forceinline__ void load_sym(const float *part, int ks, int k, double *W) {
  const int64_t kk = (int64_t)k * k;
  sum_partials<E>(part, ks, kk, [&](int64_t t, double v) {
    const int i = (int)(t / k), j = (int)(t - (int64_t)i * k);
    W[(int64_t)j * k + i] = v;
  });
  __syncthreads();
  for (int64_t t = threadIdx.x; t < kk; t += blockDim.x) {
    const int i = (int)(t / k), j = (int)(t - (int64_t)i * k);
    if (i < j) {
      const double v = 0.5 * (W[(int64_t)j * k + i] + W[(int64_t)i * k + j]);
      W[(int64_t)j * k + i] = v;
      W[(int64_t)i * k + j] = v;
    }
  }
}

// sorted eigenpairs from the orthogonalised columns (norms[] filled)
__device__ __forceinline__ void rr_emit(const double *W, const double *norms, int *perm, int k, float *V,
                        float *theta) {
  const int tid = threadIdx.x, nt = blockDim.x;
  for (int j = tid; j < k; j += nt) {
    const double v = norms[j];
    int rank = 0;
    for (int l = 0; l < k; ++l) {
      const double u = norms[l];
      rank += (u > v) || (u == v && l < j);
    }
    theta[rank] = (float)v;
    perm[rank] = j;
  }
  __syncthreads();
  const int64_t kk = (int64_t)k * k;
  for (int64_t t = tid; t < kk; t += nt) {
    const int c = (int)(t / k), i = (int)(t - (int64_t)c * k);
    const int src = perm[c];
    const double nv = norms[src];
    V[(int64_t)i * k + c] = (float)(W[(int64_t)src * k + i] * (nv > 0.0 ? 1.0 / nv : 0.0));
  }
}

// LDS eigensolver, k <= 128: 64 pairs x 16 lanes (1024 threads).  Lane l16
// of pair group g holds rows ((e + g) mod nb) * 16 + l16 of both columns in
// slot e (nb = ceil(k / 16) blocks of 16 rows), so the four pairs of a wave
// read four different row blocks at every slot.  Sweeps stop after the first
// one whose largest rotated |<p,q>| / (|p| |q|) is at most kJacobiLast: the
// next sweep would leave only about its square (far below the float32 noise
// of B) and rotate nothing the codec can see.
constexpr int kEigThreads = 1024;
constexpr double kJacobiLast = 1e-6;
__global__ __launch_bounds__(kEigThreads) void rr_eig_lds_kernel(const SmallJob *jobs,
                                                                 int max_sweeps) {
  __shared__ double W[kLdsK * kLdsK];
  __shared__ double zpad[16], sink[16];   // loads of masked slots / their stores
  __shared__ double norms[kLdsK];
  __shared__ int perm[kLdsK];
  __shared__ int any_rot, any_big;
  const SmallJob J = jobs[blockIdx.x];
  const int k = J.k, tid = threadIdx.x;
  if (tid < 16) zpad[tid] = 0.0;
  load_sym<8>(J.part, J.ks, k, W);
  __syncthreads();
  const int kp = (k + 1) & ~1, npairs = kp / 2;
  const int pi = tid >> 4, l16 = tid & 15, gw = (tid >> 4) & 3;
  const int nb = (k + 15) >> 4;
  int rows[8];
  bool rv[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    rows[e] = e < nb ? ((e + gw) % nb) * 16 + l16 : 0;
    rv[e] = e < nb && rows[e] < k;
  }
  const double tol2 = kJacobiTol * kJacobiTol, last2 = kJacobiLast * kJacobiLast;
  for (int sweep = 0; sweep < max_sweeps; ++sweep) {
    if (tid == 0) {
      any_rot = 0;
      any_big = 0;
    }
    __syncthreads();
    for (int round = 0; round < kp - 1; ++round) {
      int p = 0, q = 0;
      bool valid = pi < npairs;
      if (valid) {
        rr_pair(round, pi, kp, p, q);
        valid = q < k;
      }
      double *cp = W + p * k, *cq = W + q * k;
      double a[8], b[8];
      double alpha = 0.0, beta = 0.0, gamma = 0.0;
      // unconditional loads: a masked slot reads zeros from zpad (guarded
      // loads would each wait for the one before)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const bool ok = valid && rv[e];
        a[e] = *(ok ? cp + rows[e] : zpad + l16);
        b[e] = *(ok ? cq + rows[e] : zpad + l16);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        alpha += a[e] * a[e];
        beta += b[e] * b[e];
        gamma += a[e] * b[e];
      }
      alpha = row16_sum(alpha);
      beta = row16_sum(beta);
      gamma = row16_sum(gamma);
      // |gamma| > tol sqrt(alpha beta), squared (alpha, beta >= 0)
      if (valid && gamma != 0.0 && gamma * gamma > tol2 * (alpha * beta)) {
        double c, s;
        jacobi_cs(alpha, beta, gamma, c, s);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          *(rv[e] ? cp + rows[e] : sink + l16) = c * a[e] - s * b[e];
          *(rv[e] ? cq + rows[e] : sink + l16) = s * a[e] + c * b[e];
        }
        if (l16 == 0) {
          any_rot = 1;
          if (gamma * gamma > last2 * (alpha * beta)) any_big = 1;
        }
      }
      __syncthreads();
    }
    const int rotated = any_rot, big = any_big;
    __syncthreads();
    if (!rotated || !big) break;
  }
  for (int c = pi; c < k; c += kEigThreads / 16) {
    double s = 0.0;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const double v = *(rv[e] ? W + c * k + rows[e] : zpad + l16);
      s += v * v;
    }
    s = row16_sum(s);
    if (l16 == 0) norms[c] = sqrt(s);
  }
  __syncthreads();
  rr_emit(W, norms, perm, k, J.out, J.theta);
}

// Global-memory eigensolver for k > 128 (same ordering, rotations and stop
// rule as the LDS one): up to k = 256 each lane loads its elements of a
// column pair into registers together, then rotates them from there; past
// that it re-reads the columns.
__global__ __launch_bounds__(kSmallThreads) void rr_eig_global_kernel(const SmallJob *jobs,
                                                                      int max_sweeps) {
  __shared__ int any_rot, any_big;
  __shared__ int perm_dummy[1];
  (void)perm_dummy;
  const SmallJob J = jobs[blockIdx.x];
  const int k = J.k, tid = threadIdx.x, nt = blockDim.x;
  double *W = J.W;
  double *norms = J.aux;
  int *perm = reinterpret_cast<int *>(J.aux + k);
  load_sym<8>(J.part, J.ks, k, W);
  __syncthreads();
  const int kp = (k + 1) & ~1, npairs = kp / 2;
  const int l16 = tid & 15, groups = nt / 16;
  const double last2 = kJacobiLast * kJacobiLast;
  for (int sweep = 0; sweep < max_sweeps; ++sweep) {
    if (tid == 0) {
      any_rot = 0;
      any_big = 0;
    }
    __syncthreads();
    for (int round = 0; round < kp - 1; ++round) {
      for (int pb = 0; pb < npairs; pb += groups) {
        const int pi = pb + tid / 16;
        int p = 0, q = 0;
        bool valid = pi < npairs;
        if (valid) {
          rr_pair(round, pi, kp, p, q);
          valid = q < k;
        }
        double alpha = 0.0, beta = 0.0, gamma = 0.0;
        double *cp = W + (int64_t)p * k, *cq = W + (int64_t)q * k;
        if (k <= 16 * kEigRegs) {
          // the lane's elements of both columns loaded together into registers
          // (one round trip, not one per element), the same sums in the same
          // order, and the rotation from the registers
          double va[kEigRegs], vb[kEigRegs];
#pragma unroll
          for (int u = 0; u < kEigRegs; ++u) {
            const int i = l16 + 16 * u;
            va[u] = valid && i < k ? cp[i] : 0.0;
            vb[u] = valid && i < k ? cq[i] : 0.0;
          }
#pragma unroll
          for (int u = 0; u < kEigRegs; ++u)
            if (l16 + 16 * u < k) {
              alpha += va[u] * va[u];
              beta += vb[u] * vb[u];
              gamma += va[u] * vb[u];
            }
          alpha = row16_sum(alpha);
          beta = row16_sum(beta);
          gamma = row16_sum(gamma);
          if (valid && gamma != 0.0 && fabs(gamma) > kJacobiTol * sqrt(alpha * beta)) {
            double c, s;
            jacobi_cs(alpha, beta, gamma, c, s);
#pragma unroll
            for (int u = 0; u < kEigRegs; ++u) {
              const int i = l16 + 16 * u;
              if (i < k) {
                cp[i] = c * va[u] - s * vb[u];
                cq[i] = s * va[u] + c * vb[u];
              }
            }
            if (l16 == 0) {
              any_rot = 1;
              if (gamma * gamma > last2 * (alpha * beta)) any_big = 1;
            }
          }
        } else {
          if (valid) {
            for (int i = l16; i < k; i += 16) {
              const double a = cp[i], b = cq[i];
              alpha += a * a;
              beta += b * b;
              gamma += a * b;
            }
          }
          alpha = row16_sum(alpha);
          beta = row16_sum(beta);
          gamma = row16_sum(gamma);
          if (valid && gamma != 0.0 && fabs(gamma) > kJacobiTol * sqrt(alpha * beta)) {
            double c, s;
            jacobi_cs(alpha, beta, gamma, c, s);
            for (int i = l16; i < k; i += 16) {
              const double a = cp[i], b = cq[i];
              cp[i] = c * a - s * b;
              cq[i] = s * a + c * b;
            }
            if (l16 == 0) {
              any_rot = 1;
              if (gamma * gamma > last2 * (alpha * beta)) any_big = 1;
            }
          }
        }
        __syncthreads();
      }
    }
    const int rotated = any_rot, big = any_big;
    __syncthreads();
    if (!rotated || !big) break;
  }
  for (int c = tid / 16; c < k; c += groups) {
    double s = 0.0;
    for (int i = l16; i < k; i += 16) s += W[(int64_t)c * k + i] * W[(int64_t)c * k + i];
    s = row16_sum(s);
    if (l16 == 0) norms[c] = sqrt(s);
  }
  __syncthreads();
  rr_emit(W, norms, perm, k, J.out, J.theta);
}

// sigma^2 and the coefficients of every member (one workgroup each)
__global__ __launch_bounds__(256) void finalize_coef_kernel(const Member *mem) {
  __shared__ double red[2][4];
  const Member M = mem[blockIdx.x];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  double tr = 0.0, top = 0.0;
  for (int64_t i = tid; i < M.dim; i += 256) tr += (double)M.A[i * M.dim + i];
  for (int i = tid; i < M.r; i += 256) top += M.theta[i] > 0.f ? (double)M.theta[i] : 0.0;
  for (int o = 32; o > 0; o >>= 1) {
    tr += __shfl_xor(tr, o);
    top += __shfl_xor(top, o);
  }
  if (lane == 0) {
    red[0][wave] = tr;
    red[1][wave] = top;
  }
  __syncthreads();
  tr = (red[0][0] + red[0][1]) + (red[0][2] + red[0][3]);
  top = (red[1][0] + red[1][1]) + (red[1][2] + red[1][3]);
  const bool identity = !(tr > 0.0) || M.r == 0;
  const double floor = (double)M.damping * tr / (double)M.dim;
  double sigma2 = 0.0;
  if (!identity) {
    if (M.r >= M.dim) {
      sigma2 = tr / (double)M.dim;
    } else {
      sigma2 = (tr - top) / (double)(M.dim - M.r);
      if (sigma2 < floor) sigma2 = floor;
    }
  }
  for (int i = tid; i < M.r; i += 256) {
    double l = M.theta[i] > 0.f ? (double)M.theta[i] : 0.0;
    double cf = 0.0, ci = 0.0;
    if (!identity) {
      const double fl = M.r >= M.dim ? floor : sigma2;
      if (l < fl) l = fl;
      cf = sqrt(sigma2 / l) - 1.0;
      ci = sqrt(l / sigma2) - 1.0;
    }
    M.c_fwd[i] = (float)cf;
    M.c_inv[i] = (float)ci;
    M.lam[i] = (float)l;
  }
  if (tid == 0) M.sigma2[0] = (float)sigma2;
}

// Layouts of every member from its rotated basis (grid.y = member): Qt (all k
// rows, the warm start), Ut (first r rows), and U, U diag(c_fwd),
// U diag(c_inv) as [dim, r] through an LDS transpose of 32-row tiles.
constexpr int kTileRows = 32;
__global__ __launch_bounds__(256) void finalize_layout_kernel(const Member *mem) {
  __shared__ float tile[kLdsK][kTileRows + 1];
  const Member M = mem[blockIdx.y];
  const int tid = threadIdx.x;
  const int64_t ntiles = (M.dim + kTileRows - 1) / kTileRows;
  for (int64_t tb = blockIdx.x; tb < ntiles; tb += gridDim.x) {
    const int64_t i0 = tb * kTileRows;
    const int rows = (int)(M.dim - i0 < kTileRows ? M.dim - i0 : kTileRows);
    // copies of this column slab: Qt[a][i0..) for all k rows, Ut for a < r
    for (int t = tid; t < M.k * kTileRows; t += 256) {
      const int a = t / kTileRows, ii = t % kTileRows;
      if (ii < rows) {
        const float v = M.rot[(int64_t)a * M.dim + i0 + ii];
        M.Qt[(int64_t)a * M.dim + i0 + ii] = v;
        if (a < M.r) M.Ut[(int64_t)a * M.dim + i0 + ii] = v;
      }
    }
    for (int a0 = 0; a0 < M.r; a0 += kLdsK) {
      const int ac = M.r - a0 < kLdsK ? M.r - a0 : kLdsK;
      __syncthreads();
      for (int t = tid; t < ac * kTileRows; t += 256) {
        const int a = t / kTileRows, ii = t % kTileRows;
        tile[a][ii] = ii < rows ? M.rot[(int64_t)(a0 + a) * M.dim + i0 + ii] : 0.f;
      }
      __syncthreads();
      for (int t = tid; t < ac * rows; t += 256) {
        const int ii = t / ac, a = t % ac;
        const float u = tile[a][ii];
        const int64_t o = (i0 + ii) * M.r + a0 + a;
        M.U[o] = u;
        M.Uc[o] = u * M.c_fwd[a0 + a];
        M.Uci[o] = u * M.c_inv[a0 + a];
      }
    }
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

namespace {

// One (dim, r) group of the refresh and its slices of the workspace.
struct Group {
  std::vector<SideJob> jobs;
  int64_t dim = 0;
  int k = 0, r = 0, ks = 0, G = 0, first = 0;
  bool bf16_direct = false;
  float *Amat = nullptr, *Qw = nullptr, *Y = nullptr, *part = nullptr;
  float *Rinv = nullptr, *V = nullptr, *theta = nullptr, *Xc = nullptr;
  double *Wg = nullptr, *aux = nullptr;
  const void **xtab = nullptr;
};

}  // namespace

bool statistics_direct(gift_dtype dtype, int64_t dim) { return dtype == GIFT_BF16 && dim % 8 == 0; }

gift_status launch_statistics(gift_ctx *ctx, const void *const *d_xtab, const void *const *h_x, int G,
                              int64_t T, int64_t dim, gift_dtype dtype, float *A, float *Xc) {
  const float inv_T = (float)(1.0 / (double)T);
  gift_status st;
  if (statistics_direct(dtype, dim))
    return launch_syrk_bf16(ctx, reinterpret_cast<const uint16_t *const *>(d_xtab), G, T, dim, inv_T, A);
  for (int m = 0; m < G; ++m) {
    const float *X32 = static_cast<const float *>(h_x[m]);
    if (dtype == GIFT_BF16) {
      {
        ProfileScope prof(ctx, GIFT_KERNEL_SYRK);
        hipLaunchKernelGGL(bf16_to_f32_kernel, dim3(grid_for(T * dim)), dim3(256), 0, ctx->stream, Xc,
                           static_cast<const uint16_t *>(h_x[m]), T * dim);
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
    j.C = A + (int64_t)m * dim * dim;
    j.ldc = dim;
    j.alpha = inv_T;
    j.kernel_family = GIFT_KERNEL_SYRK;
    if ((st = launch_tile(ctx, j)) != GIFT_OK) return st;
  }
  return GIFT_OK;
}

gift_status factor_refresh_batch(gift_ctx *ctx, const std::vector<SideJob> &jobs, int64_t T,
                                 gift_dtype dtype, int32_t iters) {
  // groups in launch order: LDS-sized k first, so the small-kernel tables
  // split into one LDS range and one global range
  std::map<std::tuple<bool, int64_t, int>, Group> by_key;
  for (const SideJob &j : jobs) {
    if (j.side->r <= 0) continue;
    Group &g = by_key[std::make_tuple(j.side->k > kLdsK, j.side->dim, (int)j.side->r)];
    g.jobs.push_back(j);
  }
  if (by_key.empty()) return GIFT_OK;
  std::vector<Group> groups;
  int total = 0, n_lds = 0;
  bool any_cold = false;
  int64_t max_kd = 0;
  for (auto &kv : by_key) {
    Group g = std::move(kv.second);
    const Side &s0 = *g.jobs[0].side;
    g.dim = s0.dim;
    g.k = s0.k;
    g.r = s0.r;
    g.ks = (int)((g.dim + 255) / 256);   // split-K factor of the k x k products
    g.G = (int)g.jobs.size();
    g.first = total;
    g.bf16_direct = statistics_direct(dtype, g.dim);
    total += g.G;
    if (g.k <= kLdsK) n_lds += g.G;
    for (const SideJob &j : g.jobs) any_cold = any_cold || !j.side->have_basis || j.side->fill_tail;
    max_kd = std::max<int64_t>(max_kd, (int64_t)g.k * g.dim);
    groups.push_back(std::move(g));
  }

  // workspace: tables, then the buffers of every group (Qw and Y of all
  // groups contiguous so one copy moves them)
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align256(bytes);
    return o;
  };
  const size_t o_mem = take(sizeof(Member) * total);
  const size_t o_chol = take(sizeof(SmallJob) * total);
  const size_t o_eig = take(sizeof(SmallJob) * total);
  const size_t o_xt = take(sizeof(void *) * total);
  const size_t tables_bytes = off;
  size_t qy_floats = 0;
  for (const Group &g : groups) qy_floats += (size_t)g.G * g.k * g.dim;
  const size_t o_Q = take(sizeof(float) * qy_floats);
  const size_t o_Y = take(sizeof(float) * qy_floats);
  std::vector<size_t> o_A(groups.size()), o_P(groups.size()), o_R(groups.size()), o_V(groups.size()),
      o_th(groups.size()), o_W(groups.size()), o_aux(groups.size()), o_X(groups.size());
  for (size_t gi = 0; gi < groups.size(); ++gi) {
    const Group &g = groups[gi];
    const size_t G = g.G, k = g.k, dim = g.dim;
    o_A[gi] = take(sizeof(float) * G * dim * dim);
    o_P[gi] = take(sizeof(float) * G * g.ks * k * k);
    o_R[gi] = take(sizeof(float) * G * k * k);
    o_V[gi] = take(sizeof(float) * G * k * k);
    o_th[gi] = take(sizeof(float) * G * k);
    o_W[gi] = k > (size_t)kLdsK ? take(sizeof(double) * G * k * (k + 1)) : 0;
    o_aux[gi] = k > (size_t)kLdsK ? take(sizeof(double) * G * (2 * k + 64)) : 0;
    o_X[gi] = (dtype == GIFT_BF16 && !g.bf16_direct) ? take(sizeof(float) * (size_t)T * dim) : 0;
  }
  void *base = nullptr;
  gift_status st = workspace(ctx, off, &base);
  if (st != GIFT_OK) return st;
  char *b = static_cast<char *>(base);
  Member *d_mem = reinterpret_cast<Member *>(b + o_mem);
  SmallJob *d_chol = reinterpret_cast<SmallJob *>(b + o_chol);
  SmallJob *d_eig = reinterpret_cast<SmallJob *>(b + o_eig);
  const void **d_xt = reinterpret_cast<const void **>(b + o_xt);
  hipStream_t stream = ctx->stream;

  // host image of the tables, uploaded (through the context's pinned
  // buffer) only when it differs from the last refresh's on this context
  std::vector<char> host(tables_bytes, 0);
  Member *h_mem = reinterpret_cast<Member *>(host.data() + o_mem);
  SmallJob *h_chol = reinterpret_cast<SmallJob *>(host.data() + o_chol);
  SmallJob *h_eig = reinterpret_cast<SmallJob *>(host.data() + o_eig);
  const void **h_xt = reinterpret_cast<const void **>(host.data() + o_xt);
  size_t qy = 0;
  for (size_t gi = 0; gi < groups.size(); ++gi) {
    Group &g = groups[gi];
    const int64_t kd = (int64_t)g.k * g.dim, k2 = (int64_t)g.k * g.k;
    g.Amat = reinterpret_cast<float *>(b + o_A[gi]);
    g.Qw = reinterpret_cast<float *>(b + o_Q) + qy;
    g.Y = reinterpret_cast<float *>(b + o_Y) + qy;
    qy += (size_t)g.G * kd;
    g.part = reinterpret_cast<float *>(b + o_P[gi]);
    g.Rinv = reinterpret_cast<float *>(b + o_R[gi]);
    g.V = reinterpret_cast<float *>(b + o_V[gi]);
    g.theta = reinterpret_cast<float *>(b + o_th[gi]);
    g.Wg = o_W[gi] ? reinterpret_cast<double *>(b + o_W[gi]) : nullptr;
    g.aux = o_aux[gi] ? reinterpret_cast<double *>(b + o_aux[gi]) : nullptr;
    g.Xc = o_X[gi] ? reinterpret_cast<float *>(b + o_X[gi]) : nullptr;
    g.xtab = d_xt + g.first;
    for (int m = 0; m < g.G; ++m) {
      const Side &s = *g.jobs[m].side;
      Member &M = h_mem[g.first + m];
      M.Qt = s.Qt;
      M.Ut = s.Ut;
      M.U = s.U;
      M.Uc = s.Uc;
      M.Uci = s.Uci;
      M.c_fwd = s.c_fwd;
      M.c_inv = s.c_inv;
      M.lam = s.lam;
      M.sigma2 = s.sigma2;
      M.A = g.Amat + (int64_t)m * g.dim * g.dim;
      M.start = g.Qw + (int64_t)m * kd;
      M.rot = g.Y + (int64_t)m * kd;
      M.theta = g.theta + (int64_t)m * g.k;
      M.dim = g.dim;
      M.k = g.k;
      M.r = g.r;
      M.seed_lo = (uint32_t)(g.jobs[m].seed & 0xffffffffu);
      M.seed_hi = (uint32_t)(g.jobs[m].seed >> 32);
      M.mode = !s.have_basis ? 0 : (s.fill_tail ? 2 : 1);
      M.damping = g.jobs[m].damping;
      SmallJob &C = h_chol[g.first + m];
      C.part = g.part + (int64_t)m * g.ks * k2;
      C.out = g.Rinv + (int64_t)m * k2;
      C.theta = nullptr;
      C.W = g.Wg ? g.Wg + (int64_t)m * g.k * (g.k + 1) : nullptr;
      C.aux = g.aux ? g.aux + (int64_t)m * (2 * g.k + 64) : nullptr;
      C.ks = g.ks;
      C.k = g.k;
      SmallJob &E = h_eig[g.first + m];
      E = C;
      E.out = g.V + (int64_t)m * k2;
      E.theta = g.theta + (int64_t)m * g.k;
      h_xt[g.first + m] = g.jobs[m].x;
    }
  }
  {
    void *tb = nullptr;
    if ((st = upload_table(ctx, TAB_REFRESH, nullptr, host.data(), tables_bytes, &tb)) != GIFT_OK) return st;
    char *t = static_cast<char *>(tb);
    d_mem = reinterpret_cast<Member *>(t + o_mem);
    d_chol = reinterpret_cast<SmallJob *>(t + o_chol);
    d_eig = reinterpret_cast<SmallJob *>(t + o_eig);
    d_xt = reinterpret_cast<const void **>(t + o_xt);
    for (Group &g : groups) g.xtab = d_xt + g.first;
  }

  // 1. statistics A_g = X_g^T X_g / T
  for (Group &g : groups) {
    std::vector<const void *> xs;
    for (const SideJob &j : g.jobs) xs.push_back(j.x);
    if ((st = launch_statistics(ctx, g.xtab, xs.data(), g.G, T, g.dim, dtype, g.Amat, g.Xc)) != GIFT_OK)
      return st;
  }
  if (ctx->stats_event) GIFT_HIP_TRY(hipEventRecord(ctx->stats_event, stream));

  // 2. start blocks of every member
  {
    ProfileScope prof(ctx, GIFT_KERNEL_FACTOR);
    hipLaunchKernelGGL(gather_start_kernel, dim3(grid_for(max_kd, 256, 2048), total), dim3(256), 0, stream,
                       d_mem);
  }
  if ((st = check_launch("gather_start_kernel")) != GIFT_OK) return st;

  // part_g[m][z] = Lt_m Rt_m^T over K slice z
  auto kk_product = [&](const Group &g, const float *Lt, const float *Rt) -> gift_status {
    const int64_t kd = (int64_t)g.k * g.dim;
    TileJob j;
    j.nseg = 1;
    j.seg[0].a = Operand{Lt, g.dim, kd, true};
    j.seg[0].b = Operand{Rt, g.dim, kd, true};
    j.seg[0].K = g.dim;
    j.M = g.k;
    j.N = g.k;
    j.batch = g.G;
    j.ksplit = g.ks;
    j.C = g.part;
    j.ldc = g.k;
    j.cbs = (int64_t)g.k * g.k;
    j.kernel_family = GIFT_KERNEL_FACTOR;
    return launch_tile(ctx, j);
  };
  // C_g = Left_g^T Qw_g-shaped product: C[a][i] = sum_c L[c][a] R[c][i]
  auto small_times_block = [&](const Group &g, const float *L, const float *R, float *C) -> gift_status {
    const int64_t kd = (int64_t)g.k * g.dim, k2 = (int64_t)g.k * g.k;
    TileJob j;
    j.nseg = 1;
    j.seg[0].a = Operand{L, g.k, k2, false};     // (a, c) = L[c][a]
    j.seg[0].b = Operand{R, g.dim, kd, false};   // (c, i) = R[c][i]
    j.seg[0].K = g.k;
    j.M = g.k;
    j.N = g.dim;
    j.batch = g.G;
    j.C = C;
    j.ldc = g.dim;
    j.cbs = kd;
    j.kernel_family = GIFT_KERNEL_FACTOR;
    return launch_tile(ctx, j);
  };
  // Y_g = Qw_g A_g  (A symmetric, so (c, i) = A[i][c] reads K-major); the
  // product runs on the bf16 matrix cores with split operands (relative error
  // ~1e-6, well inside what the iteration and Rayleigh-Ritz resolve)
  auto times_A = [&](const Group &g) -> gift_status {
    const int64_t kd = (int64_t)g.k * g.dim;
    TileJob j;
    j.nseg = 1;
    j.seg[0].a = Operand{g.Qw, g.dim, kd, true};
    j.seg[0].b = Operand{g.Amat, g.dim, g.dim * g.dim, true};
    j.seg[0].K = g.dim;
    j.M = g.k;
    j.N = g.dim;
    j.batch = g.G;
    j.C = g.Y;
    j.ldc = g.dim;
    j.cbs = kd;
    j.split3 = true;
    j.kernel_family = GIFT_KERNEL_FACTOR;
    return launch_tile(ctx, j);
  };
  auto small_launch = [&](bool eig) -> gift_status {
    ProfileScope prof(ctx, eig ? GIFT_KERNEL_EIG : GIFT_KERNEL_CHOL);
    const SmallJob *tab = eig ? d_eig : d_chol;
    if (n_lds > 0) {
      if (eig)
        hipLaunchKernelGGL(rr_eig_lds_kernel, dim3(n_lds), dim3(kEigThreads), 0, stream, tab, 40);
      else
        hipLaunchKernelGGL(chol_inv_lds_kernel, dim3(n_lds), dim3(kSmallThreads), 0, stream, tab);
    }
    if (total > n_lds) {
      if (eig)
        hipLaunchKernelGGL(rr_eig_global_kernel, dim3(total - n_lds), dim3(kSmallThreads), 0, stream,
                           tab + n_lds, 40);
      else
        hipLaunchKernelGGL(chol_inv_global_kernel, dim3(total - n_lds), dim3(kCholGlobalThreads), 0, stream,
                           tab + n_lds);
    }
    return check_launch(eig ? "rr_eig_kernel" : "chol_inv_kernel");
  };
  // one CholeskyQR pass of every group: Qw = Y R^-1 with R^T R = Y^T Y
  auto cholqr_pass = [&]() -> gift_status {
    gift_status e;
    for (const Group &g : groups)
      if ((e = kk_product(g, g.Y, g.Y)) != GIFT_OK) return e;
    if ((e = small_launch(false)) != GIFT_OK) return e;
    for (const Group &g : groups)
      if ((e = small_times_block(g, g.Rinv, g.Y, g.Qw)) != GIFT_OK) return e;
    return GIFT_OK;
  };
  float *Qw_all = reinterpret_cast<float *>(b + o_Q), *Y_all = reinterpret_cast<float *>(b + o_Y);
  auto cholqr2 = [&]() -> gift_status {
    gift_status e = cholqr_pass();
    if (e != GIFT_OK) return e;
    GIFT_HIP_TRY(hipMemcpyAsync(Y_all, Qw_all, sizeof(float) * qy_floats, hipMemcpyDeviceToDevice, stream));
    return cholqr_pass();
  };

  if (any_cold) {
    GIFT_HIP_TRY(hipMemcpyAsync(Y_all, Qw_all, sizeof(float) * qy_floats, hipMemcpyDeviceToDevice, stream));
    if ((st = cholqr2()) != GIFT_OK) return st;
  }
  for (int it = 0; it < iters; ++it) {
    for (const Group &g : groups)
      if ((st = times_A(g)) != GIFT_OK) return st;
    if ((st = cholqr2()) != GIFT_OK) return st;
  }
  // Rayleigh-Ritz: B = Qw A Qw^T, eigenpairs, rotated basis V^T Qw -> Y
  for (const Group &g : groups) {
    if ((st = times_A(g)) != GIFT_OK) return st;
    if ((st = kk_product(g, g.Qw, g.Y)) != GIFT_OK) return st;
  }
  if ((st = small_launch(true)) != GIFT_OK) return st;
  for (const Group &g : groups)
    if ((st = small_times_block(g, g.V, g.Qw, g.Y)) != GIFT_OK) return st;
  {
    ProfileScope prof(ctx, GIFT_KERNEL_FACTOR);
    hipLaunchKernelGGL(finalize_coef_kernel, dim3(total), dim3(256), 0, stream, d_mem);
    int64_t max_tiles = 0;
    for (const Group &g : groups) max_tiles = std::max<int64_t>(max_tiles, (g.dim + kTileRows - 1) / kTileRows);
    hipLaunchKernelGGL(finalize_layout_kernel, dim3((unsigned)std::min<int64_t>(max_tiles, 64), total),
                       dim3(256), 0, stream, d_mem);
  }
  if ((st = check_launch("finalize kernels")) != GIFT_OK) return st;
  for (const Group &g : groups)
    for (const SideJob &jb : g.jobs) {
      jb.side->have_basis = true;
      jb.side->fill_tail = false;
    }
  return GIFT_OK;
}

size_t chol_blocks_scratch(int k, int count) {
  auto a256 = [](size_t x) { return (x + 255) & ~(size_t)255; };
  size_t b = 256;
  if (k > kLdsK)
    b += a256(sizeof(double) * (size_t)count * k * (k + 1)) + a256(sizeof(double) * (size_t)count * (2 * k + 64));
  return b;
}

gift_status launch_chol_blocks(gift_ctx *ctx, const float *G, int k, int count, float *R, float *Rinv,
                               void *scratch) {
  if (count <= 0 || k <= 0) return GIFT_OK;
  auto a256 = [](size_t x) { return (x + 255) & ~(size_t)255; };
  char *p = static_cast<char *>(scratch);
  double *W = nullptr, *aux = nullptr;
  if (k > kLdsK) {
    W = reinterpret_cast<double *>(p);
    p += a256(sizeof(double) * (size_t)count * k * (k + 1));
    aux = reinterpret_cast<double *>(p);
  }
  const int64_t kk = (int64_t)k * k;
  std::vector<SmallJob> h(count);
  for (int z = 0; z < count; ++z) {
    SmallJob &J = h[z];
    J.part = G + z * kk;
    J.out = Rinv + z * kk;
    J.rout = R + z * kk;
    J.theta = nullptr;
    J.W = W ? W + (int64_t)z * k * (k + 1) : nullptr;
    J.aux = aux ? aux + (int64_t)z * (2 * k + 64) : nullptr;
    J.ks = 1;
    J.k = k;
  }
  // the job table of these blocks (the factors written, R, identify it)
  void *tab = nullptr;
  gift_status st = upload_table(ctx, TAB_CHOL_BLOCKS, R, h.data(), sizeof(SmallJob) * (size_t)count, &tab);
  if (st != GIFT_OK) return st;
  const SmallJob *d_tab = static_cast<const SmallJob *>(tab);
  ProfileScope prof(ctx, GIFT_KERNEL_CHOL);
  if (k <= kLdsK)
    hipLaunchKernelGGL(chol_inv_lds_kernel, dim3(count), dim3(kSmallThreads), 0, ctx->stream, d_tab);
  else
    hipLaunchKernelGGL(chol_inv_global_kernel, dim3(count), dim3(kCholGlobalThreads), 0, ctx->stream, d_tab);
  return check_launch("chol_blocks");
}

}  // namespace gift
