// Dequantize-accumulate over the N data-parallel ranks held on this GPU
// (eq. dp_grad_avg; Algorithm 1's AllReduce_SUM followed by Dequantize / N,
// with each rank dequantized by its own block scale).
//
// mean[e] = fl32(acc / N), acc = fl32(acc + fl32(val(q_j[e]) * s_j[block(e)]))
// for j = 0..N-1 in order.  The translation unit is compiled without FMA
// contraction, so the result is bit-for-bit the sequence above.
//
// Layout: one workgroup (256 lanes) covers 16 rows x 256 columns; lane t
// takes row t/16 and the 4-column chunks 4*(t%16) + 64*v, v = 0..3, so each
// wave-wide access is contiguous (256 B of codes, 1 KiB of output per row).
// Block scales of the tile are staged in LDS.

#include "fp8_e4m3.h"
#include "gift_internal.h"

namespace gift {
namespace {

constexpr int kRows = 16, kCols = 256, kThreads = 256;
constexpr int kMaxScales = 4096;

struct RArgs {
  const uint8_t *codes;
  const float *scales;
  float *mean;
  int64_t m, n;
  int64_t br, bc;
  int nbr, nbc;
  int N;
  int vec;
};

__global__ __launch_bounds__(kThreads) void reduce_kernel(const RArgs p) {
  __shared__ float lds_s[kMaxScales];
  const int tid = threadIdx.x;
  const int64_t i0 = (int64_t)blockIdx.y * kRows, j0 = (int64_t)blockIdx.x * kCols;
  const int64_t i1 = i0 + kRows < p.m ? i0 + kRows : p.m;
  const int64_t j1 = j0 + kCols < p.n ? j0 + kCols : p.n;
  const int64_t bi0 = i0 / p.br, bj0 = j0 / p.bc;
  const int nlbj = (int)((j1 - 1) / p.bc - bj0 + 1);
  const int nlb = (int)((i1 - 1) / p.br - bi0 + 1) * nlbj;
  const int64_t nblk = (int64_t)p.nbr * p.nbc;
  const bool staged = (int64_t)nlb * p.N <= kMaxScales;
  if (staged) {
    for (int t = tid; t < nlb * p.N; t += kThreads) {
      const int j = t / nlb, l = t % nlb;
      const int64_t bi = bi0 + l / nlbj, bj = bj0 + l % nlbj;
      lds_s[t] = p.scales[j * nblk + bi * p.nbc + bj];
    }
  }
  __syncthreads();

  const int64_t gi = i0 + tid / 16;
  if (gi >= p.m) return;
  const int q = tid % 16;
  const int64_t lbi = gi / p.br - bi0;
  const int64_t mn = p.m * p.n;
  const float fN = (float)p.N;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int64_t gj = j0 + 4 * q + 64 * v;
    if (gj >= p.n) break;
    const bool full = p.vec && gj + 3 < p.n;
    int lbl[4];
    int64_t gbl[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int64_t c = gj + e < p.n ? gj + e : p.n - 1;
      lbl[e] = (int)(lbi * nlbj + (c / p.bc - bj0));
      gbl[e] = (gi / p.br) * p.nbc + c / p.bc;
    }
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    const int64_t off = gi * p.n + gj;
    for (int j = 0; j < p.N; ++j) {
      uint32_t word;
      if (full) {
        word = *reinterpret_cast<const uint32_t *>(p.codes + j * mn + off);
      } else {
        word = 0u;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (gj + e < p.n) word |= (uint32_t)p.codes[j * mn + off + e] << (8 * e);
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float s = staged ? lds_s[j * nlb + lbl[e]] : p.scales[j * nblk + gbl[e]];
        const float val = e4m3_decode((word >> (8 * e)) & 0xffu) * s;
        acc[e] = acc[e] + val;
      }
    }
    float *out = p.mean + off;
    if (full) {
      *reinterpret_cast<float4 *>(out) =
          make_float4(acc[0] / fN, acc[1] / fN, acc[2] / fN, acc[3] / fN);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (gj + e < p.n) out[e] = acc[e] / fN;
    }
  }
}

}  // namespace

gift_status launch_reduce(gift_ctx *ctx, const uint8_t *codes, const float *scales, int32_t N,
                          int64_t m, int64_t n, BlockGeom g, float *mean) {
  if (m <= 0 || n <= 0) return GIFT_OK;
  if (stream_eligible(m, n, g, mean, codes, nullptr, nullptr))
    return launch_stream_reduce(ctx, codes, scales, N, m, n, g, mean);
  RArgs a{};
  a.codes = codes;
  a.scales = scales;
  a.mean = mean;
  a.m = m;
  a.n = n;
  a.br = g.br;
  a.bc = g.bc;
  a.nbr = g.nbr;
  a.nbc = g.nbc;
  a.N = N;
  a.vec = (n % 4 == 0) && ((reinterpret_cast<uintptr_t>(codes) & 3) == 0) &&
          ((reinterpret_cast<uintptr_t>(mean) & 15) == 0);
  ProfileScope prof(ctx, GIFT_KERNEL_REDUCE);
  dim3 grid((unsigned)((n + kCols - 1) / kCols), (unsigned)((m + kRows - 1) / kRows));
  hipLaunchKernelGGL(reduce_kernel, grid, dim3(kThreads), 0, ctx->stream, a);
  return check_launch("reduce_kernel");
}

}  // namespace gift
