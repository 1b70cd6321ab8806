// Streaming kernels of the Euclidean branch and of the rank sum.
//
// amax / quantize (Algorithm 1's Scale and Q on W itself, Sec. I amax rule)
// and the dequantize-accumulate over the N ranks held on this GPU
// (eq. dp_grad_avg; mean = fl32(acc / N), acc = fl32(acc + fl32(val * s_j)) in
// rank order, compiled without FMA contraction).
//
// Mapping: a wave owns 256 consecutive columns (lane l: columns 4l..4l+3,
// one 16-byte access per row, so a wave reads 1 KiB contiguous per row) and a
// run of consecutive rows of one rank.  A lane's scale-block column is fixed
// for the whole run and the block row changes only at multiples of
// block_rows, tracked incrementally: no integer division per element.  Block
// maxima are reduced over the G lanes that share a block (G = largest power
// of two with 4G dividing block_cols, at most 64) and flushed with one atomic
// per group and block row into one of the block's sub-slots.
//
// Requirements (checked by the launcher, otherwise the tile kernel is used):
// n and block_cols multiples of 4, 16-byte aligned float tensors, 4-byte
// aligned codes.

#include "fp8_e4m3.h"
#include "gift_internal.h"

namespace gift {
namespace {

constexpr int kThreads = 256;
constexpr int kColsPerWave = 256;

struct SArgs {
  const float *x;      // [N][m][n]
  const float *ef_in;  // residual [N][m][n] or null (read)
  float *ef;           // residual out (quantize) or null
  uint8_t *codes;      // [N][m][n]
  float *scales;       // [N][nbr][nbc]
  uint32_t *amax;      // [N][nbr][nbc]
  float *transformed;  // optional W~ out (amax pass)
  const uint32_t *raw; // quantize from raw sub-slots [N][nbr][nbc][kAmaxSlots]
  uint32_t *clear;     // words to zero (the previous encode's slot set)
  int64_t clear_words;
  float *mean;         // [m][n] (reduce)
  int m, n, N;
  int br, bc, nbr, nbc;
  int shared;
  int rows_per_wave;
  int group;           // lanes sharing a block column (power of two)
};

__device__ __forceinline__ uint32_t group_max(uint32_t v, int group) {
  for (int o = 1; o < group; o <<= 1) {
    const uint32_t u = (uint32_t)__shfl_xor((int)v, o);
    v = u > v ? u : v;
  }
  return v;
}

__device__ __forceinline__ float4 ld4(const float *p) { return *reinterpret_cast<const float4 *>(p); }

// Per-wave row run: rows [r0, r1) of rank b, columns c0 + 4 lane.
struct Run {
  int b, r0, r1, cj;
  bool cv;
};

__device__ __forceinline__ Run wave_run(const SArgs &p, bool per_rank) {
  Run w;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wid = blockIdx.y * (kThreads / 64) + wave;
  w.b = per_rank ? (int)blockIdx.z : 0;
  w.r0 = wid * p.rows_per_wave;
  w.r1 = w.r0 + p.rows_per_wave < p.m ? w.r0 + p.rows_per_wave : p.m;
  w.cj = blockIdx.x * kColsPerWave + 4 * lane;
  w.cv = w.cj < p.n;
  return w;
}

template <bool EF>
__global__ __launch_bounds__(kThreads) void stream_amax_kernel(const SArgs p) {
  const Run w = wave_run(p, true);
  if (w.r0 >= p.m) return;
  const int lane = threadIdx.x & 63;
  const int64_t mn = (int64_t)p.m * p.n;
  const int bj = w.cv ? w.cj / p.bc : 0;
  int bi = w.r0 / p.br;
  int next = (bi + 1) * p.br;
  uint32_t run = 0u;
  const int slot = (int)((((int64_t)blockIdx.z * gridDim.y + blockIdx.y) * gridDim.x + blockIdx.x) * 4 +
                         (threadIdx.x >> 6)) % kAmaxSlots;
  auto flush = [&](int bi_) {
    const uint32_t v = group_max(run, p.group);
    if ((lane & (p.group - 1)) == 0 && w.cv && v)
      atomicMax(&p.amax[(((int64_t)w.b * p.nbr + bi_) * p.nbc + bj) * kAmaxSlots + slot], v);
    run = 0u;
  };
  const float *xb = p.x + (int64_t)w.b * mn;
  int r = w.r0;
  for (; r + 3 < w.r1 && next >= r + 4; r += 4) {   // four rows in flight
    float4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t off = (int64_t)(r + u) * p.n + w.cj;
      v[u] = w.cv ? ld4(xb + off) : make_float4(0.f, 0.f, 0.f, 0.f);
      if (EF && w.cv) {
        const float4 e = ld4(p.ef_in + (int64_t)w.b * mn + off);
        v[u].x += e.x; v[u].y += e.y; v[u].z += e.z; v[u].w += e.w;
      }
      if (p.transformed && w.cv)
        *reinterpret_cast<float4 *>(p.transformed + (int64_t)w.b * mn + off) = v[u];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const uint32_t a0 = __float_as_uint(v[u].x) & 0x7fffffffu, a1 = __float_as_uint(v[u].y) & 0x7fffffffu;
      const uint32_t a2 = __float_as_uint(v[u].z) & 0x7fffffffu, a3 = __float_as_uint(v[u].w) & 0x7fffffffu;
      uint32_t m = a0 > a1 ? a0 : a1;
      m = m > a2 ? m : a2;
      m = m > a3 ? m : a3;
      run = m > run ? m : run;
    }
    if (r + 4 == next) {
      flush(bi);
      ++bi;
      next += p.br;
    }
  }
  for (; r < w.r1; ++r) {
    const int64_t off = (int64_t)r * p.n + w.cj;
    float4 v = w.cv ? ld4(xb + off) : make_float4(0.f, 0.f, 0.f, 0.f);
    if (EF && w.cv) {
      const float4 e = ld4(p.ef_in + (int64_t)w.b * mn + off);
      v.x += e.x; v.y += e.y; v.z += e.z; v.w += e.w;
    }
    if (p.transformed && w.cv) *reinterpret_cast<float4 *>(p.transformed + (int64_t)w.b * mn + off) = v;
    const uint32_t a0 = __float_as_uint(v.x) & 0x7fffffffu, a1 = __float_as_uint(v.y) & 0x7fffffffu;
    const uint32_t a2 = __float_as_uint(v.z) & 0x7fffffffu, a3 = __float_as_uint(v.w) & 0x7fffffffu;
    uint32_t m = a0 > a1 ? a0 : a1;
    m = m > a2 ? m : a2;
    m = m > a3 ? m : a3;
    run = m > run ? m : run;
    if (r + 1 == next) {
      flush(bi);
      ++bi;
      next += p.br;
    }
  }
  flush(bi);  // the block row still open (a no-op when it was just flushed)
}

// EF: write the residual R <- x - Deq(Q(x)); ADD: x = input + R first (the
// input is W itself), otherwise the input already is W~ + R.
// RAW: the block maxima come straight from the AMAX pass's sub-slots: the G
// lanes that share a block column reduce its kAmaxSlots slots (of every rank
// for a shared scale), the wave that holds the block's first row writes its
// scale, and the grid zeroes clear_words words at clear on the way.
template <bool EF, bool ADD, bool RAW>
__global__ __launch_bounds__(kThreads) void stream_quant_kernel(const SArgs p) {
  if (RAW) {
    const int64_t nthreads = (int64_t)gridDim.x * gridDim.y * gridDim.z * kThreads;
    const int64_t gt = (((int64_t)blockIdx.z * gridDim.y + blockIdx.y) * gridDim.x + blockIdx.x) * kThreads +
                       threadIdx.x;
    for (int64_t i = gt; i < p.clear_words; i += nthreads) p.clear[i] = 0u;
  }
  const Run w = wave_run(p, true);
  if (w.r0 >= p.m) return;
  const int lane = threadIdx.x & 63;
  const int64_t mn = (int64_t)p.m * p.n;
  const int64_t nblk = (int64_t)p.nbr * p.nbc;
  // lanes past column n keep to the last block column (their group's)
  const int bj = w.cv ? w.cj / p.bc : p.nbc - 1;
  int bi = w.r0 / p.br;
  int next = (bi + 1) * p.br;
  float inv = 0.f, sc = 0.f;
  // block bi's amax; with RAW every lane of the wave takes part (group sums)
  // and the lane at the block's first column writes the scale when the block
  // starts inside this wave's rows
  auto load_scale = [&]() {
    const int64_t blk = (int64_t)bi * p.nbc + bj;
    float a;
    if (RAW) {
      const int rb = p.shared ? 0 : w.b, re = p.shared ? p.N : w.b + 1;
      uint32_t m = 0u;
      for (int r = rb; r < re; ++r) {
        const uint32_t *q = p.raw + ((int64_t)r * nblk + blk) * kAmaxSlots;
        for (int s = lane & (p.group - 1); s < kAmaxSlots; s += p.group) m = q[s] > m ? q[s] : m;
      }
      m = group_max(m, p.group);
      a = __uint_as_float(m);
      if (w.cv && (int64_t)bi * p.br >= w.r0 && w.cj % p.bc == 0) p.scales[(int64_t)w.b * nblk + blk] = e4m3_scale(a);
    } else {
      a = __uint_as_float(p.amax[(int64_t)w.b * nblk + blk]);
    }
    inv = e4m3_multiplier(a);
    sc = e4m3_scale(a);
  };
  load_scale();
  const float *xb = p.x + (int64_t)w.b * mn;
  for (int r = w.r0; r < w.r1; ++r) {
    if (r == next) {
      ++bi;
      next += p.br;
      load_scale();
    }
    if (!w.cv) continue;
    const int64_t off = (int64_t)r * p.n + w.cj;
    float4 v = ld4(xb + off);
    if (EF && ADD) {
      const float4 e = ld4(p.ef_in + (int64_t)w.b * mn + off);
      v.x += e.x; v.y += e.y; v.z += e.z; v.w += e.w;
    }
    const uint32_t packed = e4m3_encode4(v.x * inv, v.y * inv, v.z * inv, v.w * inv);
    *reinterpret_cast<uint32_t *>(p.codes + (int64_t)w.b * mn + off) = packed;
    if (EF) {
      float q[4];
      e4m3_decode4(packed, q);
      *reinterpret_cast<float4 *>(p.ef + (int64_t)w.b * mn + off) =
          make_float4(v.x - q[0] * sc, v.y - q[1] * sc, v.z - q[2] * sc, v.w - q[3] * sc);
    }
  }
}

template <int NR>
__global__ __launch_bounds__(kThreads) void stream_reduce_kernel(const SArgs p) {
  const Run w = wave_run(p, false);
  if (w.r0 >= p.m || !w.cv) return;
  const int64_t mn = (int64_t)p.m * p.n;
  const int64_t nblk = (int64_t)p.nbr * p.nbc;
  const int N = NR > 0 ? NR : p.N;
  const int bj = w.cj / p.bc;
  int bi = w.r0 / p.br;
  int next = (bi + 1) * p.br;
  constexpr int kCache = NR > 0 ? NR : 16;
  float s[kCache];
  auto load_scales = [&]() {
#pragma unroll
    for (int j = 0; j < kCache; ++j)
      s[j] = j < N ? p.scales[j * nblk + (int64_t)bi * p.nbc + bj] : 0.f;
  };
  load_scales();
  const float fN = (float)N;
  for (int r = w.r0; r < w.r1; ++r) {
    if (r == next) {
      ++bi;
      next += p.br;
      load_scales();
    }
    const int64_t off = (int64_t)r * p.n + w.cj;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    if (NR > 0) {
      uint32_t word[kCache];
#pragma unroll
      for (int j = 0; j < kCache; ++j) word[j] = *reinterpret_cast<const uint32_t *>(p.codes + j * mn + off);
#pragma unroll
      for (int j = 0; j < kCache; ++j) {
        float q[4];
        e4m3_decode4(word[j], q);
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[e] = acc[e] + q[e] * s[j];
      }
    } else {
      for (int j = 0; j < N; ++j) {
        const uint32_t word = *reinterpret_cast<const uint32_t *>(p.codes + j * mn + off);
        const float sj = j < kCache ? s[j] : p.scales[j * nblk + (int64_t)bi * p.nbc + bj];
        float q[4];
        e4m3_decode4(word, q);
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[e] = acc[e] + q[e] * sj;
      }
    }
    *reinterpret_cast<float4 *>(p.mean + off) = make_float4(acc[0] / fN, acc[1] / fN, acc[2] / fN, acc[3] / fN);
  }
}

bool al16(const void *q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; }

int lane_group(int bc) {
  int g = 1;
  while (g < 64 && (bc % (8 * g)) == 0) g <<= 1;
  return g;
}

void shape_grid(SArgs &a, int batch, dim3 &grid) {
  const int64_t colw = (a.n + kColsPerWave - 1) / kColsPerWave;
  // about eight waves per SIMD over the whole launch
  const int64_t target = 8192;
  int64_t rpw = (int64_t)a.m * colw * batch / target;
  if (rpw < 4) rpw = 4;
  if (rpw > a.m) rpw = a.m;
  a.rows_per_wave = (int)rpw;
  const int64_t waves = (a.m + rpw - 1) / rpw;
  grid = dim3((unsigned)colw, (unsigned)((waves + 3) / 4), (unsigned)batch);
}

}  // namespace

bool stream_eligible(int64_t m, int64_t n, const BlockGeom &g, const void *x, const void *codes,
                     const void *a, const void *b) {
  return n % 4 == 0 && g.bc % 4 == 0 && m < (1LL << 31) && n < (1LL << 31) && al16(x) &&
         (reinterpret_cast<uintptr_t>(codes) & 3) == 0 && (!a || al16(a)) && (!b || al16(b));
}

gift_status launch_stream_codec(gift_ctx *ctx, const TileJob &j) {
  SArgs a{};
  a.x = j.D;
  a.ef_in = j.ef;
  a.ef = j.codes ? j.ef : nullptr;
  a.codes = j.codes;
  a.scales = j.scales;
  a.amax = j.amax;
  a.transformed = j.transformed;
  a.m = (int)j.M;
  a.n = (int)j.N;
  a.N = j.batch;
  a.br = (int)j.geom.br;
  a.bc = (int)j.geom.bc;
  a.nbr = j.geom.nbr;
  a.nbc = j.geom.nbc;
  a.shared = j.shared ? 1 : 0;
  a.group = lane_group(a.bc);
  dim3 grid;
  shape_grid(a, j.batch, grid);
  ProfileScope prof(ctx, j.kernel_family);
  const bool ef = j.ef != nullptr;
  a.raw = j.from_raw ? j.amax : nullptr;
  a.clear = j.clear;
  a.clear_words = j.from_raw ? j.clear_words : 0;
  if (j.codes == nullptr) {
    if (ef) hipLaunchKernelGGL(stream_amax_kernel<true>, grid, dim3(kThreads), 0, ctx->stream, a);
    else hipLaunchKernelGGL(stream_amax_kernel<false>, grid, dim3(kThreads), 0, ctx->stream, a);
  } else if (j.from_raw) {
    if (ef && j.ef_added) hipLaunchKernelGGL((stream_quant_kernel<true, false, true>), grid, dim3(kThreads), 0, ctx->stream, a);
    else if (ef) hipLaunchKernelGGL((stream_quant_kernel<true, true, true>), grid, dim3(kThreads), 0, ctx->stream, a);
    else hipLaunchKernelGGL((stream_quant_kernel<false, false, true>), grid, dim3(kThreads), 0, ctx->stream, a);
  } else {
    if (ef && j.ef_added) hipLaunchKernelGGL((stream_quant_kernel<true, false, false>), grid, dim3(kThreads), 0, ctx->stream, a);
    else if (ef) hipLaunchKernelGGL((stream_quant_kernel<true, true, false>), grid, dim3(kThreads), 0, ctx->stream, a);
    else hipLaunchKernelGGL((stream_quant_kernel<false, false, false>), grid, dim3(kThreads), 0, ctx->stream, a);
  }
  return check_launch("stream codec kernel");
}

gift_status launch_stream_reduce(gift_ctx *ctx, const uint8_t *codes, const float *scales, int32_t N,
                                 int64_t m, int64_t n, BlockGeom g, float *mean) {
  SArgs a{};
  a.codes = const_cast<uint8_t *>(codes);
  a.scales = const_cast<float *>(scales);
  a.mean = mean;
  a.m = (int)m;
  a.n = (int)n;
  a.N = N;
  a.br = (int)g.br;
  a.bc = (int)g.bc;
  a.nbr = g.nbr;
  a.nbc = g.nbc;
  dim3 grid;
  shape_grid(a, 1, grid);
  ProfileScope prof(ctx, GIFT_KERNEL_REDUCE);
  switch (N) {
    case 4: hipLaunchKernelGGL(stream_reduce_kernel<4>, grid, dim3(kThreads), 0, ctx->stream, a); break;
    case 8: hipLaunchKernelGGL(stream_reduce_kernel<8>, grid, dim3(kThreads), 0, ctx->stream, a); break;
    case 16: hipLaunchKernelGGL(stream_reduce_kernel<16>, grid, dim3(kThreads), 0, ctx->stream, a); break;
    default: hipLaunchKernelGGL(stream_reduce_kernel<0>, grid, dim3(kThreads), 0, ctx->stream, a); break;
  }
  return check_launch("stream_reduce_kernel");
}

}  // namespace gift
