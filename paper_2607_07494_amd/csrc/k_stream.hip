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
constexpr int kGroup = 8;         // rows per load group (amax, quantize)

struct SArgs {
  const float *x;      // [N][m][n]
  const float *ef_in;  // residual [N][m][n] or null (read)
  float *ef;           // residual out (quantize) or null
  uint8_t *codes;      // [N][m][n]
  uint32_t *hits;      // quantize: boundary-hit counters [N][2] or null
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

__device__ __forceinline__ float4 ld4_if(bool ok, const float *q) {
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
  if (ok) v = ld4(q);
  return v;
}

__device__ __forceinline__ float4 add4(float4 a, const float4 &b) {
  a.x += b.x; a.y += b.y; a.z += b.z; a.w += b.w;
  return a;
}

__device__ __forceinline__ uint32_t absmax4(const float4 &v) {
  const uint32_t a0 = __float_as_uint(v.x) & 0x7fffffffu, a1 = __float_as_uint(v.y) & 0x7fffffffu;
  const uint32_t a2 = __float_as_uint(v.z) & 0x7fffffffu, a3 = __float_as_uint(v.w) & 0x7fffffffu;
  uint32_t m = a0 > a1 ? a0 : a1;
  m = m > a2 ? m : a2;
  return m > a3 ? m : a3;
}

// A wave's rows [r0, r1) go through in groups of G rows with two register
// sets: the loads of group g + 1 are issued before group g is processed, so a
// wave always has a group in flight (no single-row tail: rows past r1 are
// not loaded and not processed).
template <int G, class Set, class Load, class Proc>
__device__ __forceinline__ void row_pipeline(int r0, int r1, Set &a, Set &b, Load load, Proc proc) {
  load(r0, a);
  for (int r = r0; r < r1; r += 2 * G) {
    if (r + G < r1) load(r + G, b);
    proc(r, a);
    if (r + G >= r1) break;
    if (r + 2 * G < r1) load(r + 2 * G, a);
    proc(r + G, b);
  }
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
  const float *eb = EF ? p.ef_in + (int64_t)w.b * mn : nullptr;
  float *tb = p.transformed ? p.transformed + (int64_t)w.b * mn : nullptr;
  struct Set {
    float4 v[kGroup], e[EF ? kGroup : 1];
  };
  auto load = [&](int r, Set &s) {
#pragma unroll
    for (int u = 0; u < kGroup; ++u) {
      const bool ok = w.cv && r + u < w.r1;
      const int64_t off = (int64_t)(r + u) * p.n + w.cj;
      s.v[u] = ld4_if(ok, xb + off);
      if (EF) s.e[u] = ld4_if(ok, eb + off);
    }
  };
  auto proc = [&](int r, Set &s) {
#pragma unroll
    for (int u = 0; u < kGroup; ++u) {
      const int row = r + u;
      if (row >= w.r1) break;
      float4 x = s.v[u];
      if (EF) x = add4(x, s.e[u]);
      if (tb && w.cv) *reinterpret_cast<float4 *>(tb + (int64_t)row * p.n + w.cj) = x;
      if (row == next) {
        flush(bi);
        ++bi;
        next += p.br;
      }
      const uint32_t m = absmax4(x);
      run = m > run ? m : run;
    }
  };
  Set sa, sb;
  row_pipeline<kGroup>(w.r0, w.r1, sa, sb, load, proc);
  flush(bi);  // the block row still open
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
  uint32_t hit_up = 0u, hit_lo = 0u;
  const float *xb = p.x + (int64_t)w.b * mn;
  const float *eb = (EF && ADD) ? p.ef_in + (int64_t)w.b * mn : nullptr;
  uint8_t *cb = p.codes + (int64_t)w.b * mn;
  float *rb = EF ? p.ef + (int64_t)w.b * mn : nullptr;
  struct Set {
    float4 v[kGroup], e[(EF && ADD) ? kGroup : 1];
  };
  auto load = [&](int r, Set &s) {
#pragma unroll
    for (int u = 0; u < kGroup; ++u) {
      const bool ok = w.cv && r + u < w.r1;
      const int64_t off = (int64_t)(r + u) * p.n + w.cj;
      s.v[u] = ld4_if(ok, xb + off);
      if (EF && ADD) s.e[u] = ld4_if(ok, eb + off);
    }
  };
  auto proc = [&](int r, Set &s) {
#pragma unroll
    for (int u = 0; u < kGroup; ++u) {
      const int row = r + u;
      if (row >= w.r1) break;
      if (row == next) {
        ++bi;
        next += p.br;
        load_scale();
      }
      if (!w.cv) continue;
      float4 x = s.v[u];
      if (EF && ADD) x = add4(x, s.e[u]);
      const int64_t off = (int64_t)row * p.n + w.cj;
      const uint32_t packed = e4m3_encode4(x.x * inv, x.y * inv, x.z * inv, x.w * inv);
      *reinterpret_cast<uint32_t *>(cb + off) = packed;
      if (p.hits) e4m3_count_hits4(packed, x.x, x.y, x.z, x.w, hit_up, hit_lo);
      if (EF) {
        float q[4];
        e4m3_decode4(packed, q);
        *reinterpret_cast<float4 *>(rb + off) =
            make_float4(x.x - q[0] * sc, x.y - q[1] * sc, x.z - q[2] * sc, x.w - q[3] * sc);
      }
    }
  };
  Set sa, sb;
  row_pipeline<kGroup>(w.r0, w.r1, sa, sb, load, proc);
  if (p.hits) e4m3_flush_hits(p.hits + 2 * (int64_t)w.b, hit_up, hit_lo);
}

// Rank sum with CPL columns per lane (4: one 32-bit code word per rank and
// row; 8: one 8-byte word; 16: one 16-byte word), rows in groups of G
// pipelined as above.
template <int NR, int CPL, int G>
__global__ __launch_bounds__(kThreads) void stream_reduce_kernel(const SArgs p) {
  constexpr int W = CPL / 4;                 // 32-bit code words per rank and row
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wid = blockIdx.y * (kThreads / 64) + wave;
  const int r0 = wid * p.rows_per_wave;
  const int r1 = r0 + p.rows_per_wave < p.m ? r0 + p.rows_per_wave : p.m;
  const int cj = blockIdx.x * 64 * CPL + CPL * lane;
  if (r0 >= p.m || cj >= p.n) return;
  const int64_t mn = (int64_t)p.m * p.n;
  const int64_t nblk = (int64_t)p.nbr * p.nbc;
  const int bj = cj / p.bc;
  int bi = r0 / p.br;
  int next = (bi + 1) * p.br;
  float s[NR];
  auto load_scales = [&]() {
#pragma unroll
    for (int j = 0; j < NR; ++j) s[j] = p.scales[j * nblk + (int64_t)bi * p.nbc + bj];
  };
  load_scales();
  const float fN = (float)NR;
  struct Set {
    uint32_t c[G][NR][W];
  };
  auto load = [&](int r, Set &st) {
#pragma unroll
    for (int u = 0; u < G; ++u) {
      const bool ok = r + u < r1;
      const int64_t off = (int64_t)(r + u) * p.n + cj;
#pragma unroll
      for (int j = 0; j < NR; ++j) {
        if constexpr (W == 4) {
          uint4 v = make_uint4(0u, 0u, 0u, 0u);
          if (ok) {
            typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
            const u32x4 t = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p.codes + j * mn + off));
            v = make_uint4(t.x, t.y, t.z, t.w);
          }
          st.c[u][j][0] = v.x;
          st.c[u][j][1] = v.y;
          st.c[u][j][2] = v.z;
          st.c[u][j][3] = v.w;
        } else if constexpr (W == 2) {
          uint2 v = make_uint2(0u, 0u);
          if (ok) {
            typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
            const u32x2 t = __builtin_nontemporal_load(reinterpret_cast<const u32x2 *>(p.codes + j * mn + off));
            v = make_uint2(t.x, t.y);
          }
          st.c[u][j][0] = v.x;
          st.c[u][j][1] = v.y;
        } else {
          uint32_t v = 0u;
          if (ok) v = *reinterpret_cast<const uint32_t *>(p.codes + j * mn + off);
          st.c[u][j][0] = v;
        }
      }
    }
  };
  auto proc = [&](int r, Set &st) {
#pragma unroll
    for (int u = 0; u < G; ++u) {
      const int row = r + u;
      if (row >= r1) break;
      if (row == next) {
        ++bi;
        next += p.br;
        load_scales();
      }
      const int64_t off = (int64_t)row * p.n + cj;
#pragma unroll
      for (int q = 0; q < W; ++q) {
        float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < NR; ++j) {
          float d[4];
          e4m3_decode4(st.c[u][j][q], d);
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[e] = acc[e] + d[e] * s[j];
        }
        *reinterpret_cast<float4 *>(p.mean + off + 4 * q) =
            make_float4(acc[0] / fN, acc[1] / fN, acc[2] / fN, acc[3] / fN);
      }
    }
  };
  Set sa, sb;
  row_pipeline<G>(r0, r1, sa, sb, load, proc);
}

// any N: one row at a time, 4 columns per lane
__global__ __launch_bounds__(kThreads) void stream_reduce_any_kernel(const SArgs p) {
  const Run w = wave_run(p, false);
  if (w.r0 >= p.m || !w.cv) return;
  const int64_t mn = (int64_t)p.m * p.n;
  const int64_t nblk = (int64_t)p.nbr * p.nbc;
  const int bj = w.cj / p.bc;
  int bi = w.r0 / p.br;
  int next = (bi + 1) * p.br;
  const float fN = (float)p.N;
  for (int r = w.r0; r < w.r1; ++r) {
    if (r == next) {
      ++bi;
      next += p.br;
    }
    const int64_t off = (int64_t)r * p.n + w.cj;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int j = 0; j < p.N; ++j) {
      const uint32_t word = *reinterpret_cast<const uint32_t *>(p.codes + j * mn + off);
      const float sj = p.scales[j * nblk + (int64_t)bi * p.nbc + bj];
      float q[4];
      e4m3_decode4(word, q);
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[e] = acc[e] + q[e] * sj;
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

// rows per wave: about eight waves per SIMD over the launch, rounded up to a
// multiple of the row group `g`
void shape_grid(SArgs &a, int batch, dim3 &grid, int cols_per_wave = kColsPerWave, int g = kGroup) {
  const int64_t colw = (a.n + cols_per_wave - 1) / cols_per_wave;
  const int64_t target = 8192;
  int64_t rpw = (int64_t)a.m * colw * batch / target;
  rpw = (rpw + g - 1) / g * g;
  if (rpw < g) rpw = g;
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
  a.hits = j.codes ? j.hits : nullptr;
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
  ProfileScope prof(ctx, GIFT_KERNEL_REDUCE);
  dim3 grid;
  const bool aligned = al16(codes) && al16(mean);
  // 16 columns per lane (16-byte code words) unless 8 leave fewer lanes
  // past the last column: a wave spans 1024 columns at 16 per lane, so a
  // 1536-column matrix would leave a quarter of its lanes idle. Measured on
  // the Llama-600M set (16 ranks): rank sums 3.12 -> 2.72 ms per step in
  // isolation (4.35 -> 5.0 TB/s by (N + 4) bytes per element); one row per
  // group instead of two (more waves per SIMD) 2.61 ms alone but 5-6 ms
  // slower four-stream steps
  const auto idle = [&](int64_t cpl) { return (n + 64 * cpl - 1) / (64 * cpl) * 64 * cpl - n; };
  const bool mid = n % 8 == 0 && g.bc % 8 == 0 && aligned && idle(8) < idle(16);
  const bool wide = !mid && n % 16 == 0 && g.bc % 16 == 0 && aligned;
#define GIFT_RED(NR, CPL, G)                                                                   \
  do {                                                                                         \
    shape_grid(a, 1, grid, 64 * (CPL), (G));                                                   \
    hipLaunchKernelGGL((stream_reduce_kernel<NR, CPL, G>), grid, dim3(kThreads), 0, ctx->stream, a); \
  } while (0)
  switch (N) {
    case 4: if (wide) GIFT_RED(4, 16, 2); else if (mid) GIFT_RED(4, 8, 4); else GIFT_RED(4, 4, 4); break;
    case 8: if (wide) GIFT_RED(8, 16, 2); else if (mid) GIFT_RED(8, 8, 4); else GIFT_RED(8, 4, 4); break;
    case 16: if (wide) GIFT_RED(16, 16, 1); else if (mid) GIFT_RED(16, 8, 2); else GIFT_RED(16, 4, 2); break;
    default:
      shape_grid(a, 1, grid, kColsPerWave, 1);
      hipLaunchKernelGGL(stream_reduce_any_kernel, grid, dim3(kThreads), 0, ctx->stream, a);
      break;
  }
#undef GIFT_RED
  return check_launch("stream_reduce_kernel");
}

}  // namespace gift
