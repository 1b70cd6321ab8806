// Register-direct FP32 MFMA kernels for the codec's rank-r transform.
//
// Both kernels keep every operand in registers: no LDS staging, no barriers
// in the main loop.  A wave owns a strip of 16 rows of one rank's matrix and
// computes its block of the product transposed, so that the
// v_mfma_f32_16x16x4_f32 result puts four consecutive columns of one row in
// each lane (lane (fr, fg) holds row fr, columns 4fg..4fg+3 of each 16-column
// group).  Each lane also supplies its MFMA operands as 16-byte vectors: the
// four k values a lane feeds into four consecutive MFMA steps are four
// consecutive elements along the contraction index (any assignment of k to
// (lane group, step) gives the same sum as long as both operands use it).
//
// update_kernel: W~ = D + sum_s Row_s Col_s^T over up to two segments with
//   K_s <= 128 (the rank-r update of the forward and inverse transforms,
//   Sec. IV-A eq. design_full_transform / design_full_inverse_transform in
//   low-rank form), fused with
//     EPI_AMAX   block max |W~| (Algorithm 1's Scale): wave-reduced, one atomic
//                per wave and block into one of the block's sub-slots;
//                optional store of W~
//     EPI_QUANT  E4M3 codes with the finished block scale and the
//                error-feedback residual R <- W~ - Deq(Q(W~))
//     EPI_STORE  the inverse transform's output
// proj_kernel: out[b][i][c] = sum_k X[b][i][k] Y[c][k] (P = W U from U^T),
//   split over the contraction index across the waves of a workgroup and
//   reduced through LDS in a fixed order.

#include <type_traits>

#include "fp8_e4m3.h"
#include "gift_internal.h"
#include "xcd_map.h"

namespace gift {

static bool proj_strip_is_b(const TileJob &j);

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kMaxK16 = 8;      // K <= 128 per segment
constexpr int kColsPerUnit = 128;

struct USeg {
  const float *row;   // [batch][parts][M][K] (row_bs = 0: shared)
  int64_t row_ld, row_bs;
  int row_parts;      // split-K partials summed on load (in order)
  const float *col;   // [batch][N][K]
  int64_t col_ld, col_bs;
  int K;
  // grouped decode: batch entry b's row / column operand at row_tab[b] /
  // col_tab[b] (one partial), else as above
  const float *const *row_tab;
  const float *const *col_tab;
};

struct UArgs {
  USeg seg[2];
  int nseg;
  int64_t M, N;
  int batch;
  const float *D;       // [batch][M][N]
  float *C;             // STORE output [batch][M][N]
  uint32_t *amax;       // [batch][nbr][nbc]
  uint8_t *codes;
  uint32_t *hits;       // QUANT: boundary-hit counters [batch][2] or null
  float *scales;
  float *transformed;
  float *ef;
  int64_t br, bc;
  int nbr, nbc;
  int shared;
  const DecodePtrs *tab;  // grouped decode: per-entry column operand, D and C
  // grouped decode with both factors: per-entry D and C (the operands through
  // the segments' tables)
  const float *const *d_tab;
  float *const *c_tab;
};

__device__ __forceinline__ float4 ld4(const float *p) { return *reinterpret_cast<const float4 *>(p); }

// A 16-byte store the compiler does not track.  A store and a load in flight
// share one counter on this target, and with both kinds pending the compiler
// turns every wait for a load into a wait for everything; with this store its
// waits cover its own loads only (the hardware counter still counts the
// store, so they can only last longer).  The s_nop gives the wide store the
// wait state it needs before its data registers may be rewritten.
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void st4_untracked(float *p, float x, float y, float z, float w) {
  const u32x4_t v = {__float_as_uint(x), __float_as_uint(y), __float_as_uint(z), __float_as_uint(w)};
  asm volatile("global_store_dwordx4 %0, %1, off\n\ts_nop 1" ::"v"(p), "v"(v) : "memory");
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const uint32_t u = (uint32_t)__shfl_xor((int)v, o);
    v = u > v ? u : v;
  }
  return v;
}

// finished block amax (sub-slots and ranks already reduced)
__device__ __forceinline__ float block_amax_value(const UArgs &p, int b, int64_t gb) {
  return __uint_as_float(p.amax[(int64_t)b * p.nbr * p.nbc + gb]);
}

// One workgroup = 4 waves = 64 rows (a 16-row strip per wave) x a chunk of
// kColsPerUnit columns, walked in 64-column tiles.  The column-side operand
// of a tile (64 columns x K, shared by the 4 waves) is staged in LDS, double
// buffered: while the waves run the MFMAs of tile c, they hold the global
// loads of tile c+1's operand and of its W / residual values in registers.
template <int EPI, bool EF, int NSEG, int K16>
__global__ __launch_bounds__(kThreads) void update_kernel(const UArgs p) {
  constexpr int KT = 16 * K16 * NSEG;          // total contraction length
  constexpr int ROW = KT + 4;                  // LDS row stride (floats)
  constexpr int SLOTS = 64 * KT / 4;           // float4 slots of one tile
  constexpr int PER = SLOTS / kThreads;        // per thread (K16*NSEG)
  __shared__ __attribute__((aligned(16))) float lds[2][64 * ROW];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int fr = lane & 15, fg = lane >> 4;
  // the column units of one row block on one XCD, one after another (they
  // share the row operand)
  const int64_t lin = ((int64_t)blockIdx.z * gridDim.y + blockIdx.y) * gridDim.x + blockIdx.x;
  const int64_t wg_tile = xcd_tile(lin, (int64_t)gridDim.x * gridDim.y * gridDim.z);
  const int64_t tx = wg_tile % gridDim.x, ty = (wg_tile / gridDim.x) % gridDim.y;
  const int b = (int)(wg_tile / ((int64_t)gridDim.x * gridDim.y));
  const int64_t i0 = ty * 64 + wave * 16;
  const int64_t ri = i0 + fr;
  const bool rv = ri < p.M;
  const bool wave_live = i0 < p.M;
  const int64_t MN = p.M * p.N;
  const int64_t c_begin = tx * kColsPerUnit;
  const int slot = (int)((((int64_t)blockIdx.z * gridDim.y + blockIdx.y) * gridDim.x + blockIdx.x) * 4 + wave) %
                   kAmaxSlots;
  const int ntiles = (int)((p.N - c_begin + 63) / 64 < kColsPerUnit / 64 ? (p.N - c_begin + 63) / 64
                                                                          : kColsPerUnit / 64);

  // row-side operand fragments of the strip, kept for all column tiles: the
  // split-K partials are summed in order, one partial's fragments loaded
  // together (one round trip per partial, not one per fragment and partial)
  float4 bfr[NSEG][K16];
  const int64_t rc = rv ? ri : 0;   // rows past M read row 0 and are zeroed
#pragma unroll
  for (int s = 0; s < NSEG; ++s) {
    const int np = p.seg[s].row_parts;
    const float *base = (p.seg[s].row_tab ? p.seg[s].row_tab[b] : p.seg[s].row + (int64_t)b * np * p.seg[s].row_bs) +
                        rc * p.seg[s].row_ld + 4 * fg;
#pragma unroll
    for (int q = 0; q < K16; ++q) bfr[s][q] = ld4(base + 16 * q);
    for (int z = 1; z < np; ++z) {
      float4 u[K16];
#pragma unroll
      for (int q = 0; q < K16; ++q) u[q] = ld4(base + (int64_t)z * p.seg[s].row_bs + 16 * q);
#pragma unroll
      for (int q = 0; q < K16; ++q) {
        bfr[s][q].x += u[q].x;
        bfr[s][q].y += u[q].y;
        bfr[s][q].z += u[q].z;
        bfr[s][q].w += u[q].w;
      }
    }
#pragma unroll
    for (int q = 0; q < K16; ++q)
      if (!rv) bfr[s][q] = make_float4(0.f, 0.f, 0.f, 0.f);
  }

  // cooperative load of a column tile's operand: slot -> (column, k quad)
  float4 creg[PER];
  auto load_cols = [&](int64_t j0) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int slot = tid + u * kThreads;
      const int col = slot / (KT / 4), kq = slot % (KT / 4);
      const int s = (4 * kq) / (16 * K16), kk = 4 * kq - s * 16 * K16;
      const int64_t cj = j0 + col;
      // clamped address, unconditional load; columns past N are zeroed when
      // the tile goes to LDS
      const float *colb = p.seg[s].col_tab ? p.seg[s].col_tab[b]
                          : p.tab        ? p.tab[b].uci
                                         : p.seg[s].col + (int64_t)b * p.seg[s].col_bs;
      creg[u] = ld4(colb + (cj < p.N ? cj : 0) * p.seg[s].col_ld + kk);
    }
  };
  auto store_cols = [&](int buf, int64_t j0) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int slot = tid + u * kThreads;
      const int col = slot / (KT / 4), kq = slot % (KT / 4);
      *reinterpret_cast<float4 *>(&lds[buf][col * ROW + 4 * kq]) =
          j0 + col < p.N ? creg[u] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  // W (and residual) by unconditional buffer loads over this rank's slice:
  // rows past M read zeros, columns past N are left out by the epilogue
  const float *Db = p.d_tab ? p.d_tab[b] : p.tab ? p.tab[b].mean : p.D + (int64_t)b * MN;
  float *Cb = p.c_tab ? p.c_tab[b] : p.tab ? p.tab[b].out : (p.C ? p.C + (int64_t)b * MN : nullptr);
  const __amdgpu_buffer_rsrc_t rsD =
      __builtin_amdgcn_make_buffer_rsrc((void *)Db, (short)0, (int)(MN * 4), 0x00020000);
  const __amdgpu_buffer_rsrc_t rsE = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(EF ? p.ef + (int64_t)b * MN : p.D), (short)0, EF ? (int)(MN * 4) : 0, 0x00020000);
  const uint32_t roff = rv ? (uint32_t)(ri * p.N * 4) : 0x80000000u;
  float4 d[4], rr[4];
  auto load_w = [&](int64_t j0) {
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const uint32_t off = roff + (uint32_t)((j0 + 16 * t + 4 * fg) * 4);
      d[t] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rsD, (int)off, 0, 0));
      if (EF) rr[t] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rsE, (int)off, 0, 0));
    }
  };

  uint32_t run_max = 0u;
  int64_t run_blk = -1;
  uint32_t hit_up = 0u, hit_lo = 0u;   // QUANT boundary hits of this lane
  load_cols(c_begin);
  load_w(c_begin);
  store_cols(0, c_begin);
  __syncthreads();
  for (int ct = 0; ct < ntiles; ++ct) {
    const int buf = ct & 1;
    const int64_t j0 = c_begin + 64 * ct;
    const bool more = ct + 1 < ntiles;
    float4 dcur[4], rcur[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      dcur[t] = d[t];
      if (EF) rcur[t] = rr[t];
    }
    if (more) {
      load_cols(j0 + 64);
      load_w(j0 + 64);
    }
    floatx4 acc[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < NSEG; ++s)
#pragma unroll
      for (int q = 0; q < K16; ++q) {
        const float4 bb = bfr[s][q];
        float4 a[4];
#pragma unroll
        for (int t = 0; t < 4; ++t)
          a[t] = *reinterpret_cast<const float4 *>(
              &lds[buf][(16 * t + fr) * ROW + s * 16 * K16 + 16 * q + 4 * fg]);
        // independent accumulators back to back, so the matrix pipe overlaps them
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[t].x, bb.x, acc[t], 0, 0, 0);
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[t].y, bb.y, acc[t], 0, 0, 0);
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[t].z, bb.z, acc[t], 0, 0, 0);
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[t].w, bb.w, acc[t], 0, 0, 0);
      }
    if (more) store_cols(buf ^ 1, j0 + 64);

    if (wave_live) {
      // lane holds W~[ri][j0 + 16t + 4fg + v] = d + acc[t][v] (+ residual)
      float w[4][4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        w[t][0] = dcur[t].x + acc[t][0];
        w[t][1] = dcur[t].y + acc[t][1];
        w[t][2] = dcur[t].z + acc[t][2];
        w[t][3] = dcur[t].w + acc[t][3];
        if (EF) {
          w[t][0] += rcur[t].x;
          w[t][1] += rcur[t].y;
          w[t][2] += rcur[t].z;
          w[t][3] += rcur[t].w;
        }
      }
      if (EPI == EPI_STORE) {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int64_t cj = j0 + 16 * t + 4 * fg;
          if (rv && cj < p.N) st4_untracked(Cb + ri * p.N + cj, w[t][0], w[t][1], w[t][2], w[t][3]);
        }
      } else {
        // scale-block geometry of this wave tile (wave-uniform, two divisions)
        const int64_t rlast = (i0 + 15 < p.M ? i0 + 15 : p.M - 1);
        const int64_t clast = (j0 + 63 < p.N ? j0 + 63 : p.N - 1);
        const int bi_lo = __builtin_amdgcn_readfirstlane((int)(i0 / p.br));
        const int bj_lo = __builtin_amdgcn_readfirstlane((int)(j0 / p.bc));
        const bool uniform = (int64_t)(bi_lo + 1) * p.br > rlast && (int64_t)(bj_lo + 1) * p.bc > clast;
        const int64_t u_gb = (int64_t)bi_lo * p.nbc + bj_lo;
        if (EPI == EPI_AMAX) {
          if (p.transformed) {
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              const int64_t cj = j0 + 16 * t + 4 * fg;
              if (rv && cj < p.N)
                *reinterpret_cast<float4 *>(p.transformed + (int64_t)b * MN + ri * p.N + cj) =
                    make_float4(w[t][0], w[t][1], w[t][2], w[t][3]);
            }
          }
          if (uniform) {
            uint32_t m = 0u;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              const int64_t cj = j0 + 16 * t + 4 * fg;
              if (rv && cj < p.N) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                  const uint32_t a = __float_as_uint(w[t][e]) & 0x7fffffffu;
                  m = a > m ? a : m;
                }
              }
            }
            m = wave_max_u32(m);
            const int64_t blk = u_gb;
            if (blk != run_blk) {
              if (run_blk >= 0 && lane == 0 && run_max)
                atomicMax(&p.amax[((int64_t)b * p.nbr * p.nbc + run_blk) * kAmaxSlots + slot], run_max);
              run_blk = blk;
              run_max = 0u;
            }
            run_max = m > run_max ? m : run_max;
          } else {
            // a block edge cuts the tile: per element
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              const int64_t cj = j0 + 16 * t + 4 * fg;
              if (!(rv && cj < p.N)) continue;
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const uint32_t a = __float_as_uint(w[t][e]) & 0x7fffffffu;
                const int64_t gb = (ri / p.br) * p.nbc + (cj + e) / p.bc;
                if (a) atomicMax(&p.amax[((int64_t)b * p.nbr * p.nbc + gb) * kAmaxSlots + slot], a);
              }
            }
          }
        } else {  // EPI_QUANT
          float u_inv = 0.f, u_s = 0.f;
          if (uniform) {
            const float a = block_amax_value(p, b, u_gb);
            u_inv = e4m3_multiplier(a);
            u_s = e4m3_scale(a);
          }
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const int64_t cj = j0 + 16 * t + 4 * fg;
            if (!(rv && cj < p.N)) continue;
            uint32_t packed = 0u;
            float res[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              float inv = u_inv, sc = u_s;
              if (!uniform) {
                const float a = block_amax_value(p, b, (ri / p.br) * p.nbc + (cj + e) / p.bc);
                inv = e4m3_multiplier(a);
                sc = e4m3_scale(a);
              }
              const uint32_t code = e4m3_encode(w[t][e] * inv);
              packed |= code << (8 * e);
              if (p.hits) {
                hit_up += (code & 0x7fu) == 0x7eu;
                hit_lo += ((code & 0x7fu) == 0u) & (w[t][e] != 0.0f);
              }
              if (EF) res[e] = w[t][e] - e4m3_decode(code) * sc;
            }
            const int64_t off = (int64_t)b * MN + ri * p.N + cj;
            *reinterpret_cast<uint32_t *>(p.codes + off) = packed;
            if (EF) *reinterpret_cast<float4 *>(p.ef + off) = make_float4(res[0], res[1], res[2], res[3]);
          }
        }
      }
    }
    __syncthreads();
  }
  if (EPI == EPI_AMAX && wave_live && run_blk >= 0 && lane == 0 && run_max)
    atomicMax(&p.amax[((int64_t)b * p.nbr * p.nbc + run_blk) * kAmaxSlots + slot], run_max);
  if (EPI == EPI_QUANT && p.hits) e4m3_flush_hits(p.hits + 2 * (int64_t)b, hit_up, hit_lo);
}

struct PArgs {
  const float *X;     // [batch][M][K]
  int64_t x_ld, x_bs;
  const float *Y;     // [batch][C][K] (y_bs = 0: shared)
  int64_t y_ld, y_bs;
  int64_t M, K;
  int C;
  float *out;         // [batch][M][C], or [batch][C][M] when out_t
  int64_t out_ld, out_bs;
  int out_t;
  const DecodePtrs *tab;  // grouped decode: per-entry X (mean) and Y (U^T)
};

// KS waves of a workgroup share one 16-row strip and split K; 4 / KS strips
// per workgroup.  NT = 16-column tiles of the output per wave (C <= 16 NT).
template <int KS, int NT>
__global__ __launch_bounds__(kThreads) void proj_kernel(const PArgs p) {
  __shared__ float red[kThreads / 64][NT][64][4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int fr = lane & 15, fg = lane >> 4;
  const int b = blockIdx.z;
  const int strip = wave / KS, part = wave % KS;
  const int64_t i0 = ((int64_t)blockIdx.y * (4 / KS) + strip) * 16;
  const int c0 = blockIdx.x * 16 * NT;
  const int64_t ri = i0 + fr;
  const bool rv = ri < p.M;
  const float *xrow = p.X + (int64_t)b * p.x_bs + ri * p.x_ld;
  const float *yb = p.Y + (int64_t)b * p.y_bs;
  const int64_t nk16 = (p.K + 15) / 16;
  const int64_t per = (nk16 + KS - 1) / KS;
  const int64_t qb = part * per, qe = qb + per < nk16 ? qb + per : nk16;
  floatx4 acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
  auto fetch = [&](int64_t q, float4 &xb, float4 (&ya)[NT]) {
    const int64_t k = 16 * q + 4 * fg;
    const bool kv = k < p.K;
    xb = (rv && kv) ? ld4(xrow + k) : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int c = c0 + 16 * t + fr;
      ya[t] = (kv && c < p.C) ? ld4(yb + (int64_t)c * p.y_ld + k) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  float4 xb0, ya0[NT], xb1, ya1[NT];
  if (qb < qe) fetch(qb, xb0, ya0);
  for (int64_t q = qb; q < qe; q += 2) {
    if (q + 1 < qe) fetch(q + 1, xb1, ya1);
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(ya0[t].x, xb0.x, acc[t], 0, 0, 0);
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(ya0[t].y, xb0.y, acc[t], 0, 0, 0);
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(ya0[t].z, xb0.z, acc[t], 0, 0, 0);
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(ya0[t].w, xb0.w, acc[t], 0, 0, 0);
    if (q + 1 >= qe) break;
    if (q + 2 < qe) fetch(q + 2, xb0, ya0);
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(ya1[t].x, xb1.x, acc[t], 0, 0, 0);
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(ya1[t].y, xb1.y, acc[t], 0, 0, 0);
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(ya1[t].z, xb1.z, acc[t], 0, 0, 0);
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(ya1[t].w, xb1.w, acc[t], 0, 0, 0);
  }
  if (KS > 1) {
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int v = 0; v < 4; ++v) red[wave][t][lane][v] = acc[t][v];
    __syncthreads();
    if (part != 0) return;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        float sum = acc[t][v];
#pragma unroll
        for (int o = 1; o < KS; ++o) sum += red[wave + o][t][lane][v];
        acc[t][v] = sum;
      }
  }
  if (!rv) return;
  // lane holds out[ri][c0 + 16t + 4fg + v]
  if (p.out_t) {
    // transposed: 16 lanes of equal fg write 16 consecutive rows ri of column c
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int c = c0 + 16 * t + 4 * fg + v;
        if (c < p.C) p.out[(int64_t)b * p.out_bs + (int64_t)c * p.out_ld + ri] = acc[t][v];
      }
    return;
  }
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int c = c0 + 16 * t + 4 * fg;
    if (c < p.C)
      *reinterpret_cast<float4 *>(p.out + (int64_t)b * p.out_bs + ri * p.out_ld + c) =
          make_float4(acc[t][0], acc[t][1], acc[t][2], acc[t][3]);
  }
}

// Projection with the short operand staged in LDS: out[z][b][i][c] =
// sum_{k in part z} X[b][i][k] Y[c][k] for C = 16 NT columns.  A workgroup
// is four 16-row strips (one per wave) of one rank and one contraction part
// (blockIdx.y); the 16 NT x 64 chunk of Y for the next 64 contraction steps
// is loaded by the whole workgroup while the waves run the current one, and
// each wave holds the next chunk's X values in registers.  Sharing Y through
// LDS cuts the L2 requests for it by the four strips, which otherwise bound
// this skinny product.
template <int NT>
__global__ __launch_bounds__(kThreads) void proj_staged_kernel(const PArgs p, int parts) {
  constexpr int C = 16 * NT;
  constexpr int KC = 64;                // contraction steps per chunk
  constexpr int LD = KC + 4;            // padded LDS row (floats)
  constexpr int PER = C * KC / 4 / kThreads;   // float4 per thread per chunk (NT)
  __shared__ __attribute__((aligned(16))) float ys[2][C * LD];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int fr = lane & 15, fg = lane >> 4;
  const int b = blockIdx.z, z = blockIdx.y;
  const int64_t ri = ((int64_t)blockIdx.x * 4 + wave) * 16 + fr;
  const bool rv = ri < p.M;
  const int64_t kper = ((p.K + parts - 1) / parts + KC - 1) / KC * KC;
  const int64_t k0 = z * kper, k1 = k0 + kper < p.K ? k0 + kper : p.K;
  const int nchunks = k1 > k0 ? (int)((k1 - k0 + KC - 1) / KC) : 0;
  const float *xrow = (p.tab ? p.tab[b].mean : p.X + (int64_t)b * p.x_bs) + ri * p.x_ld;
  const float *yb = p.tab ? p.tab[b].ut : p.Y + (int64_t)b * p.y_bs;
  float4 yreg[PER], xn[4];
  auto load_y = [&](int64_t kc) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int slot = tid + u * kThreads;
      const int c = slot / (KC / 4), k4 = slot % (KC / 4);
      const int64_t k = kc + 4 * k4;
      yreg[u] = (c < p.C && k < k1) ? ld4(yb + (int64_t)c * p.y_ld + k) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  auto store_y = [&](int buf) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int slot = tid + u * kThreads;
      const int c = slot / (KC / 4), k4 = slot % (KC / 4);
      *reinterpret_cast<float4 *>(&ys[buf][c * LD + 4 * k4]) = yreg[u];
    }
  };
  auto load_x = [&](int64_t kc) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int64_t k = kc + 16 * q + 4 * fg;
      xn[q] = (rv && k < k1) ? ld4(xrow + k) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  floatx4 acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
  if (nchunks > 0) {
    load_y(k0);
    load_x(k0);
    store_y(0);
  }
  __syncthreads();
  for (int ch = 0; ch < nchunks; ++ch) {
    const int buf = ch & 1;
    float4 xc[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) xc[q] = xn[q];
    const bool more = ch + 1 < nchunks;
    if (more) {
      load_y(k0 + (int64_t)(ch + 1) * KC);
      load_x(k0 + (int64_t)(ch + 1) * KC);
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      float4 ya[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t)
        ya[t] = *reinterpret_cast<const float4 *>(&ys[buf][(16 * t + fr) * LD + 16 * q + 4 * fg]);
#pragma unroll
      for (int t = 0; t < NT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(ya[t].x, xc[q].x, acc[t], 0, 0, 0);
#pragma unroll
      for (int t = 0; t < NT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(ya[t].y, xc[q].y, acc[t], 0, 0, 0);
#pragma unroll
      for (int t = 0; t < NT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(ya[t].z, xc[q].z, acc[t], 0, 0, 0);
#pragma unroll
      for (int t = 0; t < NT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(ya[t].w, xc[q].w, acc[t], 0, 0, 0);
    }
    if (more) store_y(buf ^ 1);
    __syncthreads();
  }
  if (!rv) return;
  // lane holds part z of out[ri][16t + 4fg + v]
  float *ob = p.out + ((int64_t)b * parts + z) * p.out_bs + ri * p.out_ld;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int c = 16 * t + 4 * fg;
    if (c < p.C) *reinterpret_cast<float4 *>(ob + c) = make_float4(acc[t][0], acc[t][1], acc[t][2], acc[t][3]);
  }
}

bool al16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

bool staged_eligible(const TileJob &j) {
  const Segment &g = j.seg[0];
  return !proj_strip_is_b(j) && g.b.bs == 0 && j.N % 16 == 0 && j.N <= 128 && g.K % 4 == 0 && j.ldc % 4 == 0 &&
         j.cbs % 4 == 0 && al16(j.C);
}

}  // namespace

int proj_parts(int64_t M, int64_t K, int C, int32_t batch) {
  if (C % 16 != 0 || C > 128) return 1;
  // enough waves to cover the chip about twice, each part at least 256 deep
  const int64_t waves = (M + 15) / 16 * batch;
  int parts = 1;
  while (parts < 8 && waves * parts < 2048 && K / (2 * parts) >= 256) parts *= 2;
  return parts;
}

bool proj_staged_eligible(const TileJob &j) { return proj_kernel_eligible(j) && staged_eligible(j); }

bool update_kernel_eligible(const TileJob &j) {
  if (j.N % 4 != 0 || j.nseg < 1 || j.nseg > 2) return false;
  // per-entry tables: a store with the decode's table for neither, a
  // partial-free operand behind each table, no column scales
  if (job_has_tabs(j)) {
    if (j.amax != nullptr || j.decode_tab != nullptr || j.colscale_tab != nullptr || !j.d_tab || !j.c_tab)
      return false;
    for (int s = 0; s < j.nseg; ++s)
      if ((j.seg[s].a.tab && j.seg[s].a.parts != 1) || (j.seg[s].b.tab && j.seg[s].b.parts != 1)) return false;
  }
  if (j.M * j.N >= (1LL << 29)) return false;   // one rank's slice within a 32-bit buffer range
  const int64_t K = j.seg[0].K;
  if (K != 16 && K != 32 && K != 64 && K != 128) return false;
  for (int s = 0; s < j.nseg; ++s) {
    const Segment &g = j.seg[s];
    if (!g.a.kmajor || !g.b.kmajor || g.K != K) return false;
    if (g.a.ld % 4 || g.b.ld % 4 || g.a.bs % 4 || g.b.bs % 4) return false;
    if (!al16(g.a.ptr) || !al16(g.b.ptr)) return false;
  }
  if (!al16(j.D) || (j.C && !al16(j.C)) || (!j.D && !j.d_tab) || (j.transformed && !al16(j.transformed)) ||
      (j.ef && !al16(j.ef)) || (j.codes && (reinterpret_cast<uintptr_t>(j.codes) & 3)))
    return false;
  if (j.amax == nullptr) {  // decode store: dense output, D dense
    if (j.ldc != j.N || j.cbs != j.M * j.N || j.ldd != j.N || j.dbs != j.M * j.N || j.beta != 1.f ||
        j.alpha != 1.f || j.colscale || j.ksplit > 1)
      return false;
  }
  return true;
}

gift_status launch_update(gift_ctx *ctx, const TileJob &j) {
  UArgs a{};
  for (int s = 0; s < j.nseg; ++s) {
    a.seg[s].row = j.seg[s].a.ptr;
    a.seg[s].row_ld = j.seg[s].a.ld;
    a.seg[s].row_bs = j.seg[s].a.bs;
    a.seg[s].row_parts = j.seg[s].a.parts;
    a.seg[s].col = j.seg[s].b.ptr;
    a.seg[s].col_ld = j.seg[s].b.ld;
    a.seg[s].col_bs = j.seg[s].b.bs;
    a.seg[s].K = (int)j.seg[s].K;
    a.seg[s].row_tab = j.seg[s].a.tab;
    a.seg[s].col_tab = j.seg[s].b.tab;
  }
  a.nseg = j.nseg;
  a.M = j.M;
  a.N = j.N;
  a.batch = j.batch;
  a.D = j.D;
  a.C = j.C;
  a.amax = j.amax;
  a.codes = j.codes;
  a.hits = j.codes ? j.hits : nullptr;
  a.scales = j.scales;
  a.transformed = j.transformed;
  a.ef = j.ef;
  a.br = j.geom.br > 0 ? j.geom.br : j.M;
  a.bc = j.geom.bc > 0 ? j.geom.bc : j.N;
  a.nbr = j.geom.nbr;
  a.nbc = j.geom.nbc;
  a.shared = j.shared ? 1 : 0;
  a.tab = j.decode_tab;
  a.d_tab = j.d_tab;
  a.c_tab = j.c_tab;
  ProfileScope prof(ctx, j.kernel_family);
  dim3 grid((unsigned)((j.N + kColsPerUnit - 1) / kColsPerUnit), (unsigned)((j.M + 63) / 64),
            (unsigned)j.batch);
  const int epi = j.amax == nullptr ? EPI_STORE : (j.codes == nullptr ? EPI_AMAX : EPI_QUANT);
  const bool ef = j.ef != nullptr && epi != EPI_STORE;
  const int k16 = (int)(j.seg[0].K / 16);
  auto go = [&](auto epi_c, auto ef_c, auto nseg_c, auto k16_c) {
    hipLaunchKernelGGL((update_kernel<decltype(epi_c)::value, decltype(ef_c)::value,
                                      decltype(nseg_c)::value, decltype(k16_c)::value>),
                       grid, dim3(kThreads), 0, ctx->stream, a);
  };
  auto by_k = [&](auto epi_c, auto ef_c, auto nseg_c) {
    switch (k16) {
      case 1: go(epi_c, ef_c, nseg_c, std::integral_constant<int, 1>{}); break;
      case 2: go(epi_c, ef_c, nseg_c, std::integral_constant<int, 2>{}); break;
      case 4: go(epi_c, ef_c, nseg_c, std::integral_constant<int, 4>{}); break;
      default: go(epi_c, ef_c, nseg_c, std::integral_constant<int, 8>{}); break;
    }
  };
  auto by_seg = [&](auto epi_c, auto ef_c) {
    if (j.nseg == 1) by_k(epi_c, ef_c, std::integral_constant<int, 1>{});
    else by_k(epi_c, ef_c, std::integral_constant<int, 2>{});
  };
  using T_ = std::true_type;
  using F_ = std::false_type;
  if (epi == EPI_STORE) by_seg(std::integral_constant<int, EPI_STORE>{}, F_{});
  else if (epi == EPI_AMAX) {
    if (ef) by_seg(std::integral_constant<int, EPI_AMAX>{}, T_{});
    else by_seg(std::integral_constant<int, EPI_AMAX>{}, F_{});
  } else {
    if (ef) by_seg(std::integral_constant<int, EPI_QUANT>{}, T_{});
    else by_seg(std::integral_constant<int, EPI_QUANT>{}, F_{});
  }
  return check_launch("update_kernel");
}

// The projection kernel takes its 16-row strips from the larger output
// dimension: rows of A (out[i][c] = C[i][c]) or, for a short-and-wide output,
// rows of B (out[j][i] stored transposed into C[i][j]).
static bool proj_strip_is_b(const TileJob &j) { return j.M <= 256 && j.N > j.M; }

bool proj_kernel_eligible(const TileJob &j) {
  const Segment &g = j.seg[0];
  const bool base = j.nseg == 1 && j.amax == nullptr && g.a.kmajor && g.b.kmajor && g.K % 4 == 0 &&
                    g.a.ld % 4 == 0 && g.a.bs % 4 == 0 && g.b.ld % 4 == 0 && g.b.bs % 4 == 0 &&
                    al16(g.a.ptr) && al16(g.b.ptr) && j.D == nullptr && j.colscale == nullptr &&
                    j.alpha == 1.f;
  if (!base) return false;
  if (j.ksplit > 1) return staged_eligible(j);       // partials: staged kernel only
  if (proj_strip_is_b(j)) return true;              // transposed, scalar stores
  return j.N % 4 == 0 && j.ldc % 4 == 0 && j.cbs % 4 == 0 && al16(j.C);
}

gift_status launch_proj(gift_ctx *ctx, const TileJob &j) {
  PArgs a{};
  const bool tr = proj_strip_is_b(j);
  const Operand &xs = tr ? j.seg[0].b : j.seg[0].a;   // strip side
  const Operand &ys = tr ? j.seg[0].a : j.seg[0].b;
  a.X = xs.ptr;
  a.x_ld = xs.ld;
  a.x_bs = xs.bs;
  a.Y = ys.ptr;
  a.y_ld = ys.ld;
  a.y_bs = ys.bs;
  a.M = tr ? j.N : j.M;
  a.K = j.seg[0].K;
  a.C = (int)(tr ? j.M : j.N);
  a.out = j.C;
  a.out_ld = j.ldc;
  a.out_bs = j.cbs;
  a.out_t = tr ? 1 : 0;
  a.tab = j.decode_tab;
  ProfileScope prof(ctx, j.kernel_family);
  if (staged_eligible(j)) {
    const int parts = j.ksplit > 1 ? j.ksplit : 1;
    const int nt = (int)(j.N / 16);
    const dim3 sgrid((unsigned)((a.M + 63) / 64), (unsigned)parts, (unsigned)j.batch);
#define GIFT_PROJS(NT) hipLaunchKernelGGL((proj_staged_kernel<NT>), sgrid, dim3(kThreads), 0, ctx->stream, a, parts)
    switch (nt) {
      case 1: GIFT_PROJS(1); break;
      case 2: GIFT_PROJS(2); break;
      case 3: GIFT_PROJS(3); break;
      case 4: GIFT_PROJS(4); break;
      case 5: GIFT_PROJS(5); break;
      case 6: GIFT_PROJS(6); break;
      case 7: GIFT_PROJS(7); break;
      default: GIFT_PROJS(8); break;
    }
#undef GIFT_PROJS
    return check_launch("proj_staged_kernel");
  }
  // split K over the waves of a workgroup when strips alone would not fill the GPU
  const int64_t strips = (a.M + 15) / 16 * j.batch;
  const int ks = strips >= 4096 ? 1 : (strips >= 2048 ? 2 : 4);
  const int nt = a.C <= 16 ? 1 : (a.C <= 32 ? 2 : 4);
  const int rows_per_wg = 16 * (4 / ks);
  dim3 grid((unsigned)((a.C + 16 * nt - 1) / (16 * nt)), (unsigned)((a.M + rows_per_wg - 1) / rows_per_wg),
            (unsigned)j.batch);
#define GIFT_PROJ(KS, NT) hipLaunchKernelGGL((proj_kernel<KS, NT>), grid, dim3(kThreads), 0, ctx->stream, a)
  if (ks == 1) {
    if (nt == 1) GIFT_PROJ(1, 1); else if (nt == 2) GIFT_PROJ(1, 2); else GIFT_PROJ(1, 4);
  } else if (ks == 2) {
    if (nt == 1) GIFT_PROJ(2, 1); else if (nt == 2) GIFT_PROJ(2, 2); else GIFT_PROJ(2, 4);
  } else {
    if (nt == 1) GIFT_PROJ(4, 1); else if (nt == 2) GIFT_PROJ(4, 2); else GIFT_PROJ(4, 4);
  }
#undef GIFT_PROJ
  return check_launch("proj_kernel");
}

}  // namespace gift
