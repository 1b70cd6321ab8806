// MXFP4 encode and rank sum (OCP Microscaling Formats v1.0: FP4 E2M1 elements,
// one E8M0 power-of-two scale per 32 consecutive elements of a row), the FP4
// communication format the paper leaves as future work (Sec. I; Sec. VI,
// Discussion), applied to the transformed gradient.
//
// Encode, one pass: every lane takes 8 consecutive elements (two 16-byte
// loads), so four adjacent lanes hold one 32-element block; the block
// maximum is two lane exchanges away.  Scale exponent k = floor(log2 amax) - 2
// (clamped to -127; 255 = NaN for a block holding a NaN or an infinity),
// elements y = v * 2^-k rounded to the nearest E2M1 value with ties to the
// even code and saturation at 6, by comparisons against the midpoints (exact:
// y is exact wherever a comparison can go either way).  Codes are packed two
// per byte (element 2i in the low nibble): one 4-byte store per lane.  With
// error feedback the lane also adds the residual first and writes back
// U - dequantize(codes) (exact dequantization).
//
// Rank sum: mean[e] = fl32(acc / N), acc = fl32(acc + v_j) over ranks j in
// order, v_j the exact dequantized value.
#include <math.h>

#include "gift_internal.h"
#include "mx_fp4.h"

namespace gift {
namespace {

struct MxArgs {
  const float *x;       // [N, m, n] values to encode (W~ or W)
  const float *ef_in;   // residual added first (nullable)
  float *ef;            // residual out (nullable)
  float *transformed;   // U = x (+ residual) out (nullable)
  uint8_t *codes;       // [N, m, n / 2]
  uint8_t *scales;      // [N, m, n / 32]
  int64_t groups;       // N m n / 8 (a multiple of 4)
};

__device__ __forceinline__ float4 ld4(const float *p) { return *reinterpret_cast<const float4 *>(p); }

__global__ __launch_bounds__(256) void mx_quant_kernel(const MxArgs a) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < a.groups; g += stride) {
    const int64_t e = g * 8;
    float v[8];
    {
      const float4 p = ld4(a.x + e), q = ld4(a.x + e + 4);
      v[0] = p.x; v[1] = p.y; v[2] = p.z; v[3] = p.w;
      v[4] = q.x; v[5] = q.y; v[6] = q.z; v[7] = q.w;
    }
    if (a.ef_in) {
      const float4 p = ld4(a.ef_in + e), q = ld4(a.ef_in + e + 4);
      v[0] += p.x; v[1] += p.y; v[2] += p.z; v[3] += p.w;
      v[4] += q.x; v[5] += q.y; v[6] += q.z; v[7] += q.w;
    }
    if (a.transformed) {
      *reinterpret_cast<float4 *>(a.transformed + e) = make_float4(v[0], v[1], v[2], v[3]);
      *reinterpret_cast<float4 *>(a.transformed + e + 4) = make_float4(v[4], v[5], v[6], v[7]);
    }
    float am = 0.f;
    int bad = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float t = fabsf(v[i]);
      bad |= !(t <= 3.402823466e38f);   // NaN or infinity
      am = t > am ? t : am;
    }
    // the four lanes of one 32-element block (lanes 4b .. 4b + 3)
#pragma unroll
    for (int o = 1; o < 4; o <<= 1) {
      const float u = __shfl_xor(am, o);
      am = u > am ? u : am;
      bad |= __shfl_xor(bad, o);
    }
    const int k = mx_scale_exp(am, bad);
    uint32_t packed = 0u;
    float deq[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) packed |= mx_encode(v[i], k, bad, deq[i]) << (4 * i);
    *reinterpret_cast<uint32_t *>(a.codes + e / 2) = packed;
    if ((g & 3) == 0) a.scales[e / 32] = bad ? (uint8_t)255 : (uint8_t)(k + 127);
    if (a.ef) {
      *reinterpret_cast<float4 *>(a.ef + e) =
          make_float4(v[0] - deq[0], v[1] - deq[1], v[2] - deq[2], v[3] - deq[3]);
      *reinterpret_cast<float4 *>(a.ef + e + 4) =
          make_float4(v[4] - deq[4], v[5] - deq[5], v[6] - deq[6], v[7] - deq[7]);
    }
  }
}

__global__ __launch_bounds__(256) void mx_reduce_kernel(const uint8_t *codes, const uint8_t *scales, int N,
                                                        int64_t per_rank, float *mean) {
  // per_rank = m n elements of one rank (a multiple of 32); 8 elements per lane
  const int64_t groups = per_rank / 8;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < groups; g += stride) {
    const int64_t e = g * 8;
    float acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = 0.f;
    for (int j = 0; j < N; ++j) {
      const uint32_t p = *reinterpret_cast<const uint32_t *>(codes + (int64_t)j * (per_rank / 2) + e / 2);
      const uint32_t s = scales[(int64_t)j * (per_rank / 32) + e / 32];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint32_t c = (p >> (4 * i)) & 15u;
        float d = s == 255u ? __int_as_float(0x7fc00000) : ldexpf(e2m1_val(c & 7u), (int)s - 127);
        if (c & 8u) d = -d;
        acc[i] = acc[i] + d;
      }
    }
    const float fn = (float)N;
    *reinterpret_cast<float4 *>(mean + e) = make_float4(acc[0] / fn, acc[1] / fn, acc[2] / fn, acc[3] / fn);
    *reinterpret_cast<float4 *>(mean + e + 4) = make_float4(acc[4] / fn, acc[5] / fn, acc[6] / fn, acc[7] / fn);
  }
}

unsigned grid_for(int64_t work, int threads) {
  const int64_t g = (work + threads - 1) / threads;
  return (unsigned)(g < 1 ? 1 : (g > 16384 ? 16384 : g));
}

}  // namespace

gift_status launch_mx_quant(gift_ctx *ctx, const float *x, const float *ef_in, float *ef, float *transformed,
                            uint8_t *codes, uint8_t *scales, int64_t total) {
  MxArgs a{};
  a.x = x;
  a.ef_in = ef_in;
  a.ef = ef;
  a.transformed = transformed;
  a.codes = codes;
  a.scales = scales;
  a.groups = total / 8;
  ProfileScope prof(ctx, GIFT_KERNEL_MXFP4);
  hipLaunchKernelGGL(mx_quant_kernel, dim3(grid_for(a.groups, 256)), dim3(256), 0, ctx->stream, a);
  return check_launch("mx_quant_kernel");
}

gift_status launch_mx_reduce(gift_ctx *ctx, const uint8_t *codes, const uint8_t *scales, int32_t N,
                             int64_t per_rank, float *mean) {
  ProfileScope prof(ctx, GIFT_KERNEL_REDUCE);
  hipLaunchKernelGGL(mx_reduce_kernel, dim3(grid_for(per_rank / 8, 256)), dim3(256), 0, ctx->stream, codes, scales,
                     N, per_rank, mean);
  return check_launch("mx_reduce_kernel");
}

}  // namespace gift
