// Rank-r transform of the encode on the bf16 matrix cores.
//
// The forward transform W~ = W + (W U) diag(c) U^T (Sec. IV-A, eq.
// design_input_side_transform in low-rank form; Algorithm 1's L_A step) is
// two skinny products per rank: the projection P = W U (contraction over the
// n columns of W) and the rank-r update W + P (U diag(c))^T (contraction over
// r).  Both are memory-bound once their products are cheap, so they run on
// v_mfma_f32_16x16x32_bf16 with every float32 operand x split as
//     x = hi + lo + e,  hi = bf16(x),  lo = bf16(x - hi),  |e| <= 2^-18 |x|
// (x - hi is exact in float32) and each product formed as
//     a b ~ hi_a hi_b + hi_a lo_b + lo_a hi_b
// (the omitted lo_a lo_b is below 2^-16 |a b|).  Every partial product of two
// bf16 values is exact in float32 and the MFMA sums in float32, so W~ is
// within a few 1e-6 (relative Frobenius) of the float64 transform, where a
// float32 product chain on the FP32 matrix cores would run at 1/5 of this
// rate.  The inverse transform keeps float32 products: its coefficients
// sqrt(lambda / sigma^2) - 1 amplify the operand error.
//
// MFMA layout: lane (fr, fg) = (lane % 16, lane / 16) supplies row fr and
// eight contraction steps of each operand fragment and receives rows
// 4 fg .. 4 fg + 3, column fr of the 16 x 16 result.  The products are set up
// transposed (A operand = the column side, B operand = the row side) so that a
// lane ends up with four consecutive columns of one output row.  Within a
// 32-step chunk, lane group fg feeds contraction indices 4 fg .. 4 fg + 3 and
// 16 + 4 fg .. 16 + 4 fg + 3: two 16-byte float32 loads per row, 64 contiguous
// bytes per four lanes.  Both operands use this assignment, so the sum is the
// plain dot product.
//
// Column-side operands are staged through LDS as split [chunk][column][fg]
// 16-byte entries; entry fg of column c sits at fg ^ ((c >> 2) & 3), which
// puts the 16 rows read by one 16-lane phase in distinct banks.

#include <algorithm>
#include <type_traits>

#include "fp8_e4m3.h"
#include "gift_internal.h"
#include "mx_fp4.h"
#include "xcd_map.h"

namespace gift {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ float4 ld4(const float *p) { return *reinterpret_cast<const float4 *>(p); }
__device__ __forceinline__ float4 zero4() { return make_float4(0.f, 0.f, 0.f, 0.f); }
// 16 bytes at p when ok, else zeros.  p must be a valid address either way:
// the load itself is unconditional and the zeros come from a select, because
// a load under a branch makes every later wait for loads a full one.
__device__ __forceinline__ float4 ld4_if(bool ok, const float *p) {
  const float4 v = ld4(p);
  return ok ? v : zero4();
}

// Stores the compiler does not track.  On this target a store and a load in
// flight share one counter, and the compiler, seeing both kinds pending,
// turns every wait for a load into a wait for everything; with these stores
// its waits cover its own loads only.  The hardware counter still counts the
// stores, so those waits can only last longer, never too short.  The s_nop
// gives a wide store the wait state it needs before its data registers may
// be rewritten.
__device__ __forceinline__ void st_u32_untracked(void *p, uint32_t v) {
  asm volatile("global_store_dword %0, %1, off\n\ts_nop 1" ::"v"(p), "v"(v) : "memory");
}
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void st_u128_untracked(void *p, uint4 v) {
  const u32x4_t w = {v.x, v.y, v.z, v.w};
  asm volatile("global_store_dwordx4 %0, %1, off\n\ts_nop 1" ::"v"(p), "v"(w) : "memory");
}

// hi / lo bf16 pairs of two float32 values (round to nearest even)
__device__ __forceinline__ void split2(float x, float y, uint32_t &hi, uint32_t &lo) {
  const bf16x2 h = __builtin_convertvector((floatx2){x, y}, bf16x2);
  hi = __builtin_bit_cast(uint32_t, h);
  const float hx = __uint_as_float(hi << 16), hy = __uint_as_float(hi & 0xffff0000u);
  const bf16x2 l = __builtin_convertvector((floatx2){x - hx, y - hy}, bf16x2);
  lo = __builtin_bit_cast(uint32_t, l);
}

// eight float32 values (a: steps 0-3, b: steps 4-7) -> hi and lo fragments
__device__ __forceinline__ void split8(const float4 &a, const float4 &b, uint4 &hi, uint4 &lo) {
  split2(a.x, a.y, hi.x, lo.x);
  split2(a.z, a.w, hi.y, lo.y);
  split2(b.x, b.y, hi.z, lo.z);
  split2(b.z, b.w, hi.w, lo.w);
}

__device__ __forceinline__ bf16x8 frag(const uint4 &v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ floatx4 mfma3(const uint4 &ahi, const uint4 &alo, const uint4 &bhi,
                                         const uint4 &blo, floatx4 acc) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(frag(ahi), frag(bhi), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(frag(ahi), frag(blo), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(frag(alo), frag(bhi), acc, 0, 0, 0);
  return acc;
}

__device__ __forceinline__ int lds_slot(int c, int g) { return 4 * c + (g ^ ((c >> 2) & 3)); }

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const uint32_t u = (uint32_t)__shfl_xor((int)v, o);
    v = u > v ? u : v;
  }
  return v;
}

// ---------------------------------------------------------------------------
// Projection: out[b][z][i][c] = sum_{k in part z} X[b][i][k] Y[b][c][k], c < 16 NT
// (also the subspace iteration's Q A, as (A Q^T)^T with A symmetric)
// ---------------------------------------------------------------------------

constexpr int kProjThreads = 512;   // 8 waves x 16 rows
constexpr int kProjRows = 128;
constexpr int kProjStage = 64;      // contraction steps per LDS stage (two chunks)

struct LPArgs {
  const float *X;    // [batch][M][K], row stride K
  int64_t x_bs;
  const float *Y;    // [batch][C][K] (y_bs = 0: shared by the batch)
  int64_t y_bs;
  int64_t M, K;
  float *out;        // [batch][parts][M][C], or out_t: [batch] x [C][out_ld]
  int parts;
  int64_t kper;      // contraction steps per part (multiple of kProjStage)
  int out_t;         // store transposed (parts = 1)
  int64_t out_ld, out_bs;
  // parts = 1, not transposed: out = (acc + D) * colscale, D [batch][M][C]
  // (d_bs floats apart) and colscale [C] each optional
  const float *D;
  int64_t d_bs;
  const float *colscale;
};

template <int NT>
__global__ __launch_bounds__(kProjThreads) void lr_proj_kernel(const LPArgs p) {
  constexpr int C = 16 * NT;
  constexpr int SLOTS = 2 * C * 4;                 // (chunk, column, fg) entries per stage
  constexpr int PER = (SLOTS + kProjThreads - 1) / kProjThreads;
  __shared__ uint4 yhi[2][SLOTS], ylo[2][SLOTS];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int fr = lane & 15, fg = lane >> 4;
  const int b = blockIdx.z, z = blockIdx.y;
  const int64_t ri = (int64_t)blockIdx.x * kProjRows + wave * 16 + fr;
  const bool rv = ri < p.M;
  const int64_t k0 = (int64_t)z * p.kper;
  const int64_t k1 = k0 + p.kper < p.K ? k0 + p.kper : p.K;
  const int nst = k1 > k0 ? (int)((k1 - k0 + kProjStage - 1) / kProjStage) : 0;
  const float *xrow = p.X + (int64_t)b * p.x_bs + (rv ? ri : 0) * p.K;
  const float *yb = p.Y + (int64_t)b * p.y_bs;

  // Loads of one stage at clamped (valid) addresses with no select: the
  // zeros for slots past the range are applied where the values are used,
  // so the loads of the next stage stay in flight under this stage's MFMAs.
  float4 yr[PER][2], xr[2][2];
  auto load = [&](int64_t ks) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int s = tid + u * kProjThreads;
      const int ch = s / (4 * C), c = (s >> 2) % C, g = s & 3;
      const int64_t k = ks + 32 * ch + 4 * g;
      const float *yc = yb + (int64_t)c * p.K;
      yr[u][0] = ld4(yc + (k < k1 ? k : k0));
      yr[u][1] = ld4(yc + (k + 16 < k1 ? k + 16 : k0));
    }
#pragma unroll
    for (int ch = 0; ch < 2; ++ch) {
      const int64_t k = ks + 32 * ch + 4 * fg;
      xr[ch][0] = ld4(xrow + (k < k1 ? k : k0));
      xr[ch][1] = ld4(xrow + (k + 16 < k1 ? k + 16 : k0));
    }
  };
  auto stage_y = [&](int buf, int64_t ks) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int s = tid + u * kProjThreads;
      if (s >= SLOTS) continue;
      const int ch = s / (4 * C), c = (s >> 2) % C, g = s & 3;
      const int64_t k = ks + 32 * ch + 4 * g;
      uint4 h, l;
      split8(k < k1 ? yr[u][0] : zero4(), k + 16 < k1 ? yr[u][1] : zero4(), h, l);
      yhi[buf][ch * 4 * C + lds_slot(c, g)] = h;
      ylo[buf][ch * 4 * C + lds_slot(c, g)] = l;
    }
  };

  floatx4 acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
  if (nst > 0) {
    load(k0);
    stage_y(0, k0);
  }
  __syncthreads();
  for (int st = 0; st < nst; ++st) {
    const int buf = st & 1;
    const int64_t ks = k0 + (int64_t)st * kProjStage;
    uint4 xh[2], xl[2];
#pragma unroll
    for (int ch = 0; ch < 2; ++ch) {
      const int64_t k = ks + 32 * ch + 4 * fg;
      split8(rv && k < k1 ? xr[ch][0] : zero4(), rv && k + 16 < k1 ? xr[ch][1] : zero4(), xh[ch], xl[ch]);
    }
    const bool more = st + 1 < nst;
    if (more) load(ks + kProjStage);
#pragma unroll
    for (int ch = 0; ch < 2; ++ch)
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const int e = ch * 4 * C + lds_slot(16 * t + fr, fg);
        acc[t] = mfma3(yhi[buf][e], ylo[buf][e], xh[ch], xl[ch], acc[t]);
      }
    if (more) stage_y(buf ^ 1, ks + kProjStage);
    __syncthreads();
  }
  if (!rv) return;
  // lane holds part z of out[ri][16 t + 4 fg + v]
  if (p.out_t) {
    // transposed: the 16 lanes of equal fg write 16 consecutive rows ri
    float *ob = p.out + (int64_t)b * p.out_bs + ri;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int v = 0; v < 4; ++v) ob[(int64_t)(16 * t + 4 * fg + v) * p.out_ld] = acc[t][v];
    return;
  }
  float *ob = p.out + (((int64_t)b * p.parts + z) * p.M + ri) * C;
  const float *db = p.D ? p.D + (int64_t)b * p.d_bs + ri * C : nullptr;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    float4 v = make_float4(acc[t][0], acc[t][1], acc[t][2], acc[t][3]);
    if (db) {
      const float4 d = ld4(db + 16 * t + 4 * fg);
      v.x += d.x; v.y += d.y; v.z += d.z; v.w += d.w;
    }
    if (p.colscale) {
      const float4 c = ld4(p.colscale + 16 * t + 4 * fg);
      v.x *= c.x; v.y *= c.y; v.z *= c.z; v.w *= c.w;
    }
    *reinterpret_cast<float4 *>(ob + 16 * t + 4 * fg) = v;
  }
}

// P[b][i][c] = sum_z partial[b][z][i][c], z in order (float32), so that the
// update reads one P instead of every partial once per column range
__global__ __launch_bounds__(256) void lr_psum_kernel(const float *part, float *out, int parts,
                                                      int64_t per_rank, int64_t total) {
  // per_rank = M * C floats of one rank's P, total = batch * per_rank (multiples of 4)
  const int64_t stride = (int64_t)gridDim.x * blockDim.x * 4;
  for (int64_t e = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4; e < total; e += stride) {
    const int64_t b = e / per_rank, i = e - b * per_rank;
    const float *q = part + b * parts * per_rank + i;
    float4 acc = ld4(q);
    for (int z = 1; z < parts; ++z) {
      const float4 v = ld4(q + (int64_t)z * per_rank);
      acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
    }
    *reinterpret_cast<float4 *>(out + e) = acc;
  }
}

// ---------------------------------------------------------------------------
// Update: W~[b][i][j] = D[b][i][j] + sum_s sum_k Row_s[b][i][k] Col_s[b][j][k]
//         (+ R[b][i][j]), fused with the block maxima (EPI_AMAX) or with the
//         scale, E4M3 pack and residual update (EPI_QUANT)
// ---------------------------------------------------------------------------

constexpr int kUpdThreads = 256;    // 4 waves x 32 rows
constexpr int kUpdRows = 128;
// 64-column tiles per workgroup: the column operand of all of them sits in
// LDS (8 KiB per tile and 32-step chunk), at most 64 KiB
constexpr int upd_tiles(int nch) { return nch <= 2 ? 4 : (nch <= 4 ? 2 : 1); }

struct LUSeg {
  const float *row;   // [batch][parts][M][K] (row_bs = 0: shared by the batch)
  int64_t row_ld, row_bs;
  int row_parts;      // split-K partials summed in order on load
  const float *col;   // [batch][N][K] (col_bs = 0: shared)
  int64_t col_ld, col_bs;
  int K;
};

struct LUArgs {
  LUSeg seg[2];
  int64_t M, N;
  const float *D;       // [batch][M][N]
  uint32_t *amax;       // AMAX: raw sub-slots; QUANT: finished maxima [batch][nbr][nbc]
  uint8_t *codes;
  uint32_t *hits;       // QUANT: boundary-hit counters [batch][2] or null
  float *transformed;   // AMAX: optional W~ (+ R) out
  float *ef;            // residual (read; QUANT also writes it)
  int64_t br, bc;
  int nbr, nbc;
  int codes_wide;       // N % 16 == 0 and 16-byte aligned codes: 16-byte stores
  // QUANT straight from the AMAX pass's raw sub-slots (every wave tile inside
  // one scale block): block maxima reduced in the kernel, scales written by
  // the wave holding a block's first element, clear_words words at clear
  // zeroed on the way
  const uint32_t *raw;
  float *scales;
  uint32_t *clear;
  int64_t clear_words;
  int shared, batch;
  uint8_t *mx_codes;    // MX: packed E2M1 codes [batch][M][N/2]
  uint8_t *mx_scales;   // MX: E8M0 scales [batch][M][N/32]
  int upw = 1;                      // sweep variant: 128 x 128 units per workgroup
  const void *col_img = nullptr;    // sweep variant: the column operand's LDS image
  int64_t img_bs = 0;               // bytes between batch entries' images (0: shared)
  const void *col_img2 = nullptr;   // sweep variant, two segments: segment 1's image
  int64_t img_bs2 = 0;              // bytes between batch entries' segment-1 images (0: shared)
};

template <int EPI, bool EF, int NSEG, int KC, bool FULL>
__device__ __forceinline__ void lr_update_body(const LUArgs &p) {
  static_assert(!FULL || EPI != EPI_STORE, "FULL is an AMAX / QUANT variant");
  constexpr int NCH = NSEG * KC;                // 32-step chunks over all segments
  constexpr int TSLOTS = NCH * 64 * 4;          // (chunk, column, fg) entries of a 64-column tile
  constexpr int TILES = upd_tiles(NCH);
  constexpr int COLS = 64 * TILES;
  constexpr int SLOTS = TILES * TSLOTS;         // the workgroup's whole column range
  constexpr int PER = SLOTS / kUpdThreads;      // = TILES * NCH
  __shared__ uint4 chi[SLOTS], clo[SLOTS];
  // QUANT: a wave's codes of two consecutive 32 x 64 tiles (one, when the
  // range holds one tile), written in the matrix-core layout (4 bytes per
  // lane and 16-column group) and read back as 16 consecutive codes per
  // lane: the global stores are 16 bytes wide and each row's 128 codes of a
  // tile pair leave in one instruction, whole 128-byte lines (a half line
  // would make the cache fetch the other half from HBM before merging it)
  constexpr bool PAIR = TILES >= 2;
  constexpr int CW = PAIR ? 32 : 16;            // staged words per row
  __shared__ uint32_t cstage[EPI == EPI_QUANT ? kUpdThreads / 64 : 1][32 * CW];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int fr = lane & 15, fg = lane >> 4;
  // the column units of one row block on one XCD, one after another, so
  // the row operand they share is read from HBM once
  const int64_t lin = ((int64_t)blockIdx.z * gridDim.y + blockIdx.y) * gridDim.x + blockIdx.x;
  const int64_t wg_tile = xcd_tile(lin, (int64_t)gridDim.x * gridDim.y * gridDim.z);
  const int64_t tx = wg_tile % gridDim.x, ty = (wg_tile / gridDim.x) % gridDim.y;
  const int b = (int)(wg_tile / ((int64_t)gridDim.x * gridDim.y));
  const int64_t i0 = ty * kUpdRows + wave * 32;
  const int64_t MN = p.M * p.N;
  const int64_t c_begin = tx * COLS;
  const int64_t c_end = c_begin + COLS < p.N ? c_begin + COLS : p.N;
  const int ntiles = (int)((c_end - c_begin + 63) / 64);
  const bool wave_live = i0 < p.M;
  const int slot = (int)((((int64_t)blockIdx.z * gridDim.y + blockIdx.y) * gridDim.x + blockIdx.x) * 4 + wave) %
                   kAmaxSlots;
  if (EPI == EPI_QUANT && p.clear_words) {
    const int64_t nthreads = (int64_t)gridDim.x * gridDim.y * gridDim.z * kUpdThreads;
    const int64_t gt = (((int64_t)blockIdx.z * gridDim.y + blockIdx.y) * gridDim.x + blockIdx.x) * kUpdThreads + tid;
    for (int64_t i = gt; i < p.clear_words; i += nthreads) st_u32_untracked(p.clear + i, 0u);
  }
  int64_t q_blk = -1;      // block whose maximum q_amax holds (QUANT from raw slots)
  float q_amax = 0.f;
  int64_t ri[2];
  bool rv[2];
#pragma unroll
  for (int g = 0; g < 2; ++g) {
    ri[g] = i0 + 16 * g + fr;
    rv[g] = ri[g] < p.M;
  }

  // W (and residual) values of the wave's 32 x 64 tile: lane holds row
  // ri[g], columns j0 + 16 t + 4 fg .. + 3; two register sets alternate
  typedef float4 WTile[2][4];
  // Unconditional buffer loads over this rank's M x N slice (a guarded load
  // would make every later wait a full one): rows past M fall outside the
  // range and read zeros; columns past N read the next row or zeros, and the
  // epilogue leaves them out.
  const __amdgpu_buffer_rsrc_t rsD =
      __builtin_amdgcn_make_buffer_rsrc((void *)(p.D + (int64_t)b * MN), (short)0, (int)(MN * 4), 0x00020000);
  const __amdgpu_buffer_rsrc_t rsE = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(EF ? p.ef + (int64_t)b * MN : p.D), (short)0, EF ? (int)(MN * 4) : 0, 0x00020000);
  uint32_t roff[2];
#pragma unroll
  for (int g = 0; g < 2; ++g) roff[g] = rv[g] ? (uint32_t)(ri[g] * p.N * 4) : 0x80000000u;
  auto load_w = [&](int64_t j0, WTile &dd, WTile &re) {
#pragma unroll
    for (int g = 0; g < 2; ++g)
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const uint32_t off = roff[g] + (uint32_t)((j0 + 16 * t + 4 * fg) * 4);
        dd[g][t] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rsD, (int)off, 0, 0));
        if (EF) re[g][t] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rsE, (int)off, 0, 0));
      }
  };
  // Prologue loads in the order they are needed, all unconditional so that
  // each wait covers only what it must: the column operand of the whole
  // column range and the row fragments' first partials, then the first two
  // W tiles (in flight while the operands are split into LDS).
  // FULL QUANT: the finished maximum of each tile's block from the AMAX
  // pass's raw sub-slots (lane l reads sub-slot l; every rank's when shared)
  uint32_t t_raw[TILES];
  if (FULL && EPI == EPI_QUANT) {
    const int64_t nblk = (int64_t)p.nbr * p.nbc;
    const int64_t bi = (i0 < p.M ? i0 : p.M - 1) / p.br;
#pragma unroll
    for (int ct = 0; ct < TILES; ++ct) {
      const int64_t gb = bi * p.nbc + (c_begin + 64 * ct) / p.bc;
      uint32_t m = p.raw[((int64_t)b * nblk + gb) * kAmaxSlots + lane];
      if (p.shared)
        for (int r = 0; r < p.batch; ++r) {
          const uint32_t v = p.raw[((int64_t)r * nblk + gb) * kAmaxSlots + lane];
          m = v > m ? v : m;
        }
      t_raw[ct] = m;
    }
  }
  float4 cv[PER][2];
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int s = tid + u * kUpdThreads;
    const int ct = s / TSLOTS, rem = s % TSLOTS;
    const int ch = rem / 256, c = (rem >> 2) & 63, g = rem & 3;
    const LUSeg &sg = p.seg[ch / KC];
    const int64_t k = 32 * (ch % KC) + 4 * g;
    const int64_t j = c_begin + 64 * ct + c;
    const float *q = sg.col + (int64_t)b * sg.col_bs + (j < p.N ? j : 0) * sg.col_ld;
    cv[u][0] = ld4_if(j < p.N && k < sg.K, q + (k < sg.K ? k : 0));
    cv[u][1] = ld4_if(j < p.N && k + 16 < sg.K, q + (k + 16 < sg.K ? k + 16 : 0));
  }
  float4 rv0[2][NCH], rv1[2][NCH];
#pragma unroll
  for (int g = 0; g < 2; ++g)
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
      const LUSeg &sg = p.seg[ch / KC];
      const int64_t k = 32 * (ch % KC) + 4 * fg;
      const float *q = sg.row + (int64_t)b * sg.row_parts * sg.row_bs + (rv[g] ? ri[g] : 0) * sg.row_ld;
      rv0[g][ch] = ld4_if(rv[g] && k < sg.K, q + (k < sg.K ? k : 0));
      rv1[g][ch] = ld4_if(rv[g] && k + 16 < sg.K, q + (k + 16 < sg.K ? k + 16 : 0));
    }
  WTile dA, dB, rA, rB;
  load_w(c_begin, dA, rA);
  load_w(c_begin + 64, dB, rB);   // past the range when ntiles == 1: not used
  __builtin_amdgcn_sched_barrier(0);   // keep every prologue load ahead of the first wait

  // the column operand split into LDS: entry s -> (tile, chunk, column, fg)
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int s = tid + u * kUpdThreads;
    const int ct = s / TSLOTS, rem = s % TSLOTS;
    const int ch = rem / 256, c = (rem >> 2) & 63, g = rem & 3;
    uint4 h, l;
    split8(cv[u][0], cv[u][1], h, l);
    chi[ct * TSLOTS + ch * 256 + lds_slot(c, g)] = h;
    clo[ct * TSLOTS + ch * 256 + lds_slot(c, g)] = l;
  }

  // row-side fragments of the wave's 32 rows (split-K partials summed in
  // order), split once for all tiles
  uint4 rh[2][NCH], rl[2][NCH];
#pragma unroll
  for (int g = 0; g < 2; ++g)
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
      const LUSeg &sg = p.seg[ch / KC];
      const int64_t k = 32 * (ch % KC) + 4 * fg;
      float4 v0 = rv0[g][ch], v1 = rv1[g][ch];
      if (sg.row_parts > 1) {
        const float *base = sg.row + (int64_t)b * sg.row_parts * sg.row_bs + (rv[g] ? ri[g] : 0) * sg.row_ld;
        for (int zp = 1; zp < sg.row_parts; ++zp) {
          const float *q = base + (int64_t)zp * sg.row_bs;
          const float4 a = ld4_if(rv[g] && k < sg.K, q + (k < sg.K ? k : 0));
          const float4 c = ld4_if(rv[g] && k + 16 < sg.K, q + (k + 16 < sg.K ? k + 16 : 0));
          v0.x += a.x; v0.y += a.y; v0.z += a.z; v0.w += a.w;
          v1.x += c.x; v1.y += c.y; v1.z += c.z; v1.w += c.w;
        }
      }
      split8(v0, v1, rh[g][ch], rl[g][ch]);
    }

  __syncthreads();

  uint32_t run_max = 0u;
  int64_t run_blk = -1;
  uint32_t hit_up = 0u, hit_lo = 0u;   // QUANT boundary hits of this lane
  // FULL: every wave tile lies in one scale block and the workgroup's whole
  // column range is processed without branches, so the compiler can wait for
  // one register set of W while the next one stays in flight.  AMAX keeps the
  // tiles' maxima here and merges them into the block slots after the loop
  // (no store in the loop)
  uint32_t tmax[TILES];
#pragma unroll
  for (int t = 0; t < TILES; ++t) tmax[t] = 0u;
  // one 64-column tile, no barrier: products from LDS, epilogue on `cur`,
  // then the loads of tile ct + 2 into the same register set
  auto tile = [&](int ct, WTile &cur, WTile &curR) {
    const int64_t j0 = c_begin + 64 * ct;
    floatx4 acc[2][4];
#pragma unroll
    for (int g = 0; g < 2; ++g)
#pragma unroll
      for (int t = 0; t < 4; ++t) acc[g][t] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int e = ct * TSLOTS + ch * 256 + lds_slot(16 * t + fr, fg);
        const uint4 ah = chi[e], al = clo[e];
#pragma unroll
        for (int g = 0; g < 2; ++g) acc[g][t] = mfma3(ah, al, rh[g][ch], rl[g][ch], acc[g][t]);
      }
      if (wave_live) {
        float w[2][4][4];
  #pragma unroll
        for (int g = 0; g < 2; ++g)
  #pragma unroll
          for (int t = 0; t < 4; ++t) {
            w[g][t][0] = cur[g][t].x + acc[g][t][0];
            w[g][t][1] = cur[g][t].y + acc[g][t][1];
            w[g][t][2] = cur[g][t].z + acc[g][t][2];
            w[g][t][3] = cur[g][t].w + acc[g][t][3];
            if (EF) {
              w[g][t][0] += curR[g][t].x;
              w[g][t][1] += curR[g][t].y;
              w[g][t][2] += curR[g][t].z;
              w[g][t][3] += curR[g][t].w;
            }
          }
        // scale-block geometry of the wave tile (wave-uniform, two divisions)
        const int64_t rlast = i0 + 31 < p.M ? i0 + 31 : p.M - 1;
        const int64_t clast = j0 + 63 < p.N ? j0 + 63 : p.N - 1;
        const int bi_lo = __builtin_amdgcn_readfirstlane((int)(i0 / p.br));
        const int bj_lo = __builtin_amdgcn_readfirstlane((int)(j0 / p.bc));
        const bool uniform = (int64_t)(bi_lo + 1) * p.br > rlast && (int64_t)(bj_lo + 1) * p.bc > clast;
        const int64_t u_gb = (int64_t)bi_lo * p.nbc + bj_lo;
        const int64_t nblk = (int64_t)p.nbr * p.nbc;
        if (EPI == EPI_MX) {
          // MXFP4: the lanes fr, fr + 16, fr + 32, fr + 48 hold the 32
          // columns j0 + 32 h .. of row ri[g] (8 each, in t = 2h, 2h + 1)
          const int64_t nsb = p.N / 32;
#pragma unroll
          for (int g = 0; g < 2; ++g)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              float am = 0.f;
              int bad = 0;
#pragma unroll
              for (int tt = 0; tt < 2; ++tt)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                  const float a = fabsf(w[g][2 * h + tt][e]);
                  bad |= !(a <= 3.402823466e38f);
                  am = a > am ? a : am;
                }
#pragma unroll
              for (int o = 16; o < 64; o <<= 1) {
                const float u = __shfl_xor(am, o);
                am = u > am ? u : am;
                bad |= __shfl_xor(bad, o);
              }
              const int k = mx_scale_exp(am, bad);
              const int64_t cb = j0 + 32 * h;
              const bool ok = rv[g] && cb < p.N;
#pragma unroll
              for (int tt = 0; tt < 2; ++tt) {
                const int t = 2 * h + tt;
                const int64_t cj = j0 + 16 * t + 4 * fg;
                uint32_t pk = 0u;
                float d[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) pk |= mx_encode(w[g][t][e], k, bad, d[e]) << (4 * e);
                if (ok) {
                  const int64_t off = (int64_t)b * MN + ri[g] * p.N + cj;
                  *reinterpret_cast<uint16_t *>(p.mx_codes + off / 2) = (uint16_t)pk;
                  if (EF)
                    *reinterpret_cast<float4 *>(p.ef + off) =
                        make_float4(w[g][t][0] - d[0], w[g][t][1] - d[1], w[g][t][2] - d[2], w[g][t][3] - d[3]);
                  if (p.transformed)
                    *reinterpret_cast<float4 *>(p.transformed + off) =
                        make_float4(w[g][t][0], w[g][t][1], w[g][t][2], w[g][t][3]);
                }
              }
              if (ok && fg == 0)
                p.mx_scales[((int64_t)b * p.M + ri[g]) * nsb + cb / 32] = bad ? (uint8_t)255 : (uint8_t)(k + 127);
            }
        } else if (FULL && EPI == EPI_AMAX) {
          uint32_t m = 0u;
  #pragma unroll
          for (int g = 0; g < 2; ++g)
  #pragma unroll
            for (int t = 0; t < 4; ++t) {
              const int64_t cj = j0 + 16 * t + 4 * fg;
              if (rv[g] && cj < p.N) {
  #pragma unroll
                for (int e = 0; e < 4; ++e) {
                  const uint32_t a = __float_as_uint(w[g][t][e]) & 0x7fffffffu;
                  m = a > m ? a : m;
                }
              }
            }
          tmax[ct] = wave_max_u32(m);
        } else if (EPI == EPI_AMAX) {
          if (p.transformed) {
  #pragma unroll
            for (int g = 0; g < 2; ++g)
  #pragma unroll
              for (int t = 0; t < 4; ++t) {
                const int64_t cj = j0 + 16 * t + 4 * fg;
                if (rv[g] && cj < p.N)
                  *reinterpret_cast<float4 *>(p.transformed + (int64_t)b * MN + ri[g] * p.N + cj) =
                      make_float4(w[g][t][0], w[g][t][1], w[g][t][2], w[g][t][3]);
              }
          }
          if (uniform) {
            uint32_t m = 0u;
  #pragma unroll
            for (int g = 0; g < 2; ++g)
  #pragma unroll
              for (int t = 0; t < 4; ++t) {
                const int64_t cj = j0 + 16 * t + 4 * fg;
                if (rv[g] && cj < p.N) {
  #pragma unroll
                  for (int e = 0; e < 4; ++e) {
                    const uint32_t a = __float_as_uint(w[g][t][e]) & 0x7fffffffu;
                    m = a > m ? a : m;
                  }
                }
              }
            m = wave_max_u32(m);
            if (u_gb != run_blk) {
              if (run_blk >= 0 && lane == 0 && run_max)
                atomicMax(&p.amax[((int64_t)b * nblk + run_blk) * kAmaxSlots + slot], run_max);
              run_blk = u_gb;
              run_max = 0u;
            }
            run_max = m > run_max ? m : run_max;
          } else {
            // a block edge cuts the tile: per element
  #pragma unroll
            for (int g = 0; g < 2; ++g)
  #pragma unroll
              for (int t = 0; t < 4; ++t) {
                const int64_t cj = j0 + 16 * t + 4 * fg;
                if (!(rv[g] && cj < p.N)) continue;
  #pragma unroll
                for (int e = 0; e < 4; ++e) {
                  const uint32_t a = __float_as_uint(w[g][t][e]) & 0x7fffffffu;
                  const int64_t gb = (ri[g] / p.br) * p.nbc + (cj + e) / p.bc;
                  if (a) atomicMax(&p.amax[((int64_t)b * nblk + gb) * kAmaxSlots + slot], a);
                }
              }
          }
        } else {  // EPI_QUANT with finished block maxima
          float u_inv = 0.f, u_s = 0.f;
          if (FULL) {
            const float a = __uint_as_float(wave_max_u32(t_raw[ct]));
            u_inv = e4m3_multiplier(a);
            u_s = e4m3_scale(a);
            if (lane == 0 && i0 == (int64_t)bi_lo * p.br && j0 == (int64_t)bj_lo * p.bc)
              st_u32_untracked(p.scales + (int64_t)b * nblk + u_gb, __float_as_uint(u_s));
          } else if (uniform) {
            float a;
            if (p.raw) {
              if (u_gb != q_blk) {
                // lane l reads sub-slot l of the block (of every rank when shared)
                const int r0 = p.shared ? 0 : b, r1 = p.shared ? p.batch : b + 1;
                uint32_t m = 0u;
                for (int r = r0; r < r1; ++r) {
                  const uint32_t v = p.raw[((int64_t)r * nblk + u_gb) * kAmaxSlots + lane];
                  m = v > m ? v : m;
                }
                q_amax = __uint_as_float(wave_max_u32(m));
                q_blk = u_gb;
                if (lane == 0 && i0 == (int64_t)bi_lo * p.br && j0 == (int64_t)bj_lo * p.bc)
                  st_u32_untracked(p.scales + (int64_t)b * nblk + u_gb, __float_as_uint(e4m3_scale(q_amax)));
              }
              a = q_amax;
            } else {
              a = __uint_as_float(p.amax[(int64_t)b * nblk + u_gb]);
            }
            u_inv = e4m3_multiplier(a);
            u_s = e4m3_scale(a);
          }
  #pragma unroll
          for (int g = 0; g < 2; ++g)
  #pragma unroll
            for (int t = 0; t < 4; ++t) {
              const int64_t cj = j0 + 16 * t + 4 * fg;
              if (!(rv[g] && cj < p.N)) continue;
              float inv[4] = {u_inv, u_inv, u_inv, u_inv}, sc[4] = {u_s, u_s, u_s, u_s};
              if (!FULL && !uniform) {
  #pragma unroll
                for (int e = 0; e < 4; ++e) {
                  const float a = __uint_as_float(p.amax[(int64_t)b * nblk + (ri[g] / p.br) * p.nbc + (cj + e) / p.bc]);
                  inv[e] = e4m3_multiplier(a);
                  sc[e] = e4m3_scale(a);
                }
              }
              const uint32_t packed = e4m3_encode4(w[g][t][0] * inv[0], w[g][t][1] * inv[1], w[g][t][2] * inv[2],
                                                   w[g][t][3] * inv[3]);
              if (p.hits) e4m3_count_hits4(packed, w[g][t][0], w[g][t][1], w[g][t][2], w[g][t][3], hit_up, hit_lo);
              float res[4];
              if (EF) {
                float q[4];
                e4m3_decode4(packed, q);
  #pragma unroll
                for (int e = 0; e < 4; ++e) res[e] = w[g][t][e] - q[e] * sc[e];
              }
              const int64_t off = (int64_t)b * MN + ri[g] * p.N + cj;
              cstage[wave][(16 * g + fr) * CW + (PAIR ? 16 * (ct & 1) : 0) + 4 * t + fg] = packed;
              if (EF)
                st_u128_untracked(p.ef + off, make_uint4(__float_as_uint(res[0]), __float_as_uint(res[1]),
                                                         __float_as_uint(res[2]), __float_as_uint(res[3])));
            }
          // a pair is stored after its second tile, or after a last tile
          // without a partner (its missing half lies past N)
          if (!PAIR || (ct & 1) || ct + 1 == ntiles) {
            // the wave reads back only what its own lanes wrote: the fences
            // order these LDS accesses (no workgroup barrier)
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
            const int64_t jp = PAIR ? j0 - 64 * (ct & 1) : j0;   // first column staged
            constexpr int QPR = CW / 4;                          // 16-byte chunks per row
#pragma unroll
            for (int h = 0; h < 32 * QPR / 64; ++h) {
              const int c = lane + 64 * h;         // 16-byte chunk: row c / QPR, chunk c % QPR
              const int row = c / QPR, qt = c % QPR;
              const int64_t gi = i0 + row;
              const int64_t cj = jp + 16 * qt;
              const uint4 v = *reinterpret_cast<const uint4 *>(&cstage[wave][row * CW + 4 * qt]);
              if (gi < p.M) {
                uint8_t *dst = p.codes + (int64_t)b * MN + gi * p.N + cj;
                if (FULL || (p.codes_wide && cj + 16 <= p.N)) {
                  st_u128_untracked(dst, v);
                } else {
                  const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                  for (int q = 0; q < 4; ++q)
                    if (cj + 4 * q < p.N) st_u32_untracked(dst + 4 * q, wv[q]);
                }
              }
            }
          }
        }
      }
    if (FULL ? ct + 2 < TILES : ct + 2 < ntiles) load_w(j0 + 128, cur, curR);
  };
  if (FULL) {
    // every tile of the range, also past N in the last range of an AMAX pass
    // (its maxima leave those columns out; QUANT runs FULL only when N fills
    // every range): no branch between the waits.  TILES is 1 from five
    // chunks on, so the second tile of a pair exists only when TILES > 1
    // (a compile-time test): a tile past the range would belong to the next
    // workgroup's columns.
#pragma unroll
    for (int ct = 0; ct < TILES; ct += 2) {
      tile(ct, dA, rA);
      if (ct + 1 < TILES) tile(ct + 1, dB, rB);
    }
    // one atomic per run of tiles in the same block
    if (EPI == EPI_AMAX && wave_live && lane == 0) {
      const int64_t nblk = (int64_t)p.nbr * p.nbc;
      const int64_t brow = (i0 / p.br) * p.nbc;
#pragma unroll
      for (int ct = 0; ct < TILES; ++ct) {
        if (ct >= ntiles) break;
        const int64_t gb = brow + (c_begin + 64 * ct) / p.bc;
        if (run_blk != gb) {
          if (run_blk >= 0 && run_max)
            atomicMax(&p.amax[((int64_t)b * nblk + run_blk) * kAmaxSlots + slot], run_max);
          run_blk = gb;
          run_max = tmax[ct];
        } else {
          run_max = tmax[ct] > run_max ? tmax[ct] : run_max;
        }
      }
    }
  } else {
    for (int ct = 0; ct < ntiles; ct += 2) {
      tile(ct, dA, rA);
      if (ct + 1 < ntiles) tile(ct + 1, dB, rB);
    }
  }
  if (EPI == EPI_AMAX && wave_live && run_blk >= 0 && lane == 0 && run_max)
    atomicMax(&p.amax[((int64_t)b * p.nbr * p.nbc + run_blk) * kAmaxSlots + slot], run_max);
  if (EPI == EPI_QUANT && p.hits) e4m3_flush_hits(p.hits + 2 * (int64_t)b, hit_up, hit_lo);
}

template <int EPI, bool EF, int NSEG, int KC, bool FULL = false>
__global__ __launch_bounds__(kUpdThreads) void lr_update_kernel(const LUArgs p) {
  lr_update_body<EPI, EF, NSEG, KC, FULL>(p);
}

// The same kernel held to two waves per SIMD (at most 256 VGPRs + AGPRs per
// lane).  From 128 contraction steps on (rank-128 transforms) the unbounded
// build takes one wave per SIMD, which leaves the loads of a wave's tiles
// with nothing to hide behind; two workgroups per CU still fit in LDS.
// Variants (epilogue, residual, 32-step chunks, branch-free) built for two
// waves per SIMD: 4-6 chunks without a residual, the ones that fit 256 VGPRs
// with no scratch (the branch-free AMAX pass at 4 chunks does not).
constexpr bool upd_two_waves(int epi, bool ef, int nch, bool full) {
  return epi != EPI_MX && !ef && nch >= 4 && nch <= 6 && !(epi == EPI_AMAX && full && nch == 4);
}
template <int EPI, bool EF, int NSEG, int KC, bool FULL = false>
__global__ __launch_bounds__(kUpdThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void lr_update_kernel_o2(
    const LUArgs p) {
  lr_update_body<EPI, EF, NSEG, KC, FULL>(p);
}

#define GIFT_LDS __attribute__((address_space(3)))

// s_waitcnt vmcnt(N) alone (expcnt and lgkmcnt at their maxima): at most N
// vector memory operations of this wave still outstanding
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt is six bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// A workgroup barrier for LDS written by copies that other copies still in
// flight do not touch: this wave's vector-memory operations down to N
// outstanding (its copies that must have landed) and all its LDS accesses
// done, then the barrier.  No memory fence: a workgroup-scope release would
// also wait for the copies meant to stay in flight across the barrier.  The
// empty asm statements keep the compiler from moving memory accesses across.
template <int N>
__device__ __forceinline__ void copies_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt is six bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (0 << 8));
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// The column-operand image: entry (tile T, chunk ch, column c, fg g) holds
// the hi and lo fragments of col[64 T + c][32 ch + 4 g .. + 3] and
// [32 ch + 16 + 4 g .. + 3] (split8), hi at T 2 TS + ch 256 + lds_slot(c, g)
// and lo TS entries after it, TS = 256 K / 32: the LDS layout of one tile.
// count > 1: operand b at col + b col_bs, its image 2 entries uint4 after
// operand b - 1's.
__global__ __launch_bounds__(256) void lr_col_image_kernel(const float *col, int64_t ld, int64_t col_bs,
                                                           int64_t entries, int64_t count, int nch, uint4 *img) {
  const int TS = nch * 256;
  const int64_t total = entries * count;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
    const int64_t b = i / entries, ie = i - b * entries;
    const int g = (int)(ie & 3), c = (int)((ie >> 2) & 63);
    const int64_t r = ie >> 8;
    const int ch = (int)(r % nch);
    const int64_t T = r / nch;
    const float *q = col + b * col_bs + (64 * T + c) * ld + 32 * ch + 4 * g;
    uint4 h, l;
    split8(ld4(q), ld4(q + 16), h, l);
    uint4 *o = img + b * 2 * entries + T * 2 * TS + ch * 256 + lds_slot(c, g);
    o[0] = h;
    o[TS] = l;
  }
}

// ---------------------------------------------------------------------------
// Sweep variant of the encode's two passes at rank 32 KC (64, 96, 128; N a
// multiple of 128, every 32 x 64 wave tile inside one scale block, per-rank
// scales, no boundary-hit counts): the input-side transform alone (one
// segment, with or without the error-feedback residual) or both sides at
// equal ranks (two segments, the rank-2r update, no residual).  A workgroup
// walks a run of `upw` consecutive 128 x 128 units of the batch, ordered
// (rank, row block, column pair), 64 columns at a time.  Per tile it
// multiplies from one half of a double-buffered LDS ring while the next
// tile's column operand is copied into the other half straight from its
// pre-split image (no registers, no conversions) and W of the tile after
// next is loading into the register set just consumed; the row operand (the
// rows of P) is loaded and split once per row block.  The products are those
// of lr_update_body in the same order and the image holds the same splits,
// so W~, the block maxima and the codes are bit-identical to it.  WT: the
// AMAX pass also stores W~ (both sides at rank 96 or 128, whose update is
// bound by the matrix cores: the quantize pass then streams the stored W~).
// ---------------------------------------------------------------------------

template <int EPI, int KC, bool EF, int NSEG, bool WT>
__device__ __forceinline__ void lr_sweep_body(const LUArgs &p) {
  static_assert(EPI == EPI_AMAX || EPI == EPI_QUANT, "sweep: AMAX or QUANT");
  static_assert(!WT || EPI == EPI_AMAX, "sweep: W~ stored by the AMAX pass");
  static_assert(NSEG == 1 || (NSEG == 2 && !EF), "sweep: two segments without a residual");
  constexpr int NCH = NSEG * KC;    // 32-step chunks over both segments
  // W (and the residual) of the tile after next in a second register set,
  // or, with a residual at rank 96 or 128 (whose two sets would not fit two
  // waves per SIMD), of the next tile in the one set (its loads then wait
  // behind the tile's products only)
  // With two segments (the two-sided transform's rank-2r update) the row
  // operand of both takes 128 registers, so W also loads one tile ahead,
  // and each ring half holds one segment's image: a tile multiplies
  // segment 0 from one half while segment 1 is copied into the other, then
  // segment 1 while the next tile's segment 0 is copied.
  constexpr bool DEEP = NSEG == 1 && !(EF && KC >= 3);
  constexpr int TS = KC * 256;      // (chunk, column, fg) entries of one segment's 64-column tile
  constexpr int CPW = 2 * TS / 64 / 4;   // 1-KiB pieces of a tile's image per wave
  // the two halves of the ring as separate arrays, so that the compiler's
  // wait analysis tells the copies into one from reads of the other: hi
  // fragments at [0, TS), lo at [TS, 2 TS)
  __shared__ __attribute__((aligned(1024))) uint4 ring0[2 * TS], ring1[2 * TS];
  __shared__ uint32_t cstage[EPI == EPI_QUANT ? kUpdThreads / 64 : 1][32 * 32];
  // (the wave index in a scalar register: every wave-derived offset scalar)
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int fr = lane & 15, fg = lane >> 4;
  const int64_t MN = p.M * p.N;
  const int M32 = (int)p.M, N32 = (int)p.N;
  const int ucols = N32 / 128;
  const int per_rank = (M32 + kUpdRows - 1) / kUpdRows * ucols;
  const int total = per_rank * p.batch;               // < 2^31 (launcher)
  // consecutive runs (the runs of one row block, which share its rows of P)
  // on one XCD, one after another
  const int u0 = (int)xcd_tile(blockIdx.x, gridDim.x) * p.upw;
  const int Q = 2 * ((u0 + p.upw < total ? u0 + p.upw : total) - u0);   // tiles of the run, >= 2
  const int slot = (int)(((int64_t)blockIdx.x * 4 + wave) % kAmaxSlots);
  // block indices over the batch fit 32 bits with their sub-slots (launcher)
  const int nblk = (int)(p.nbr * p.nbc);
  const int br = (int)p.br, bc = (int)p.bc;
  if (EPI == EPI_QUANT && p.clear_words) {
    const int64_t nthreads = (int64_t)gridDim.x * kUpdThreads;
    for (int64_t i = (int64_t)blockIdx.x * kUpdThreads + tid; i < p.clear_words; i += nthreads)
      st_u32_untracked(p.clear + i, 0u);
  }
  // tile q of the run: rank b, row block rb, first column j0 (wave-uniform)
  auto coord = [&](int q, int &b, int &rb, int &j0) {
    const int u = u0 + (q >> 1);
    b = u / per_rank;
    const int r = u - b * per_rank;
    rb = r / ucols;
    j0 = (r - rb * ucols) * 128 + 64 * (q & 1);
  };
  typedef float4 WTile[2][4];
  // W (and the residual) of tile q (rows past M fall outside the buffer
  // range and read zeros; so does every row of a tile past the run, q >= Q:
  // no fetch at all)
  auto load_w = [&](int q, WTile &dd, WTile &re) {
    const bool in_run = q < Q;
    int b, rb, j0;
    coord(in_run ? q : Q - 1, b, rb, j0);
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc((void *)(p.D + (int64_t)b * MN), (short)0, (int)(MN * 4), 0x00020000);
    const __amdgpu_buffer_rsrc_t rsE = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(EF ? p.ef + (int64_t)b * MN : p.D), (short)0, EF ? (int)(MN * 4) : 0, 0x00020000);
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      const int r = rb * kUpdRows + wave * 32 + 16 * g + fr;
      const uint32_t ro = in_run && r < M32 ? (uint32_t)r * (uint32_t)N32 * 4u : 0x80000000u;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int off = (int)(ro + (uint32_t)(j0 + 16 * t + 4 * fg) * 4u);
        dd[g][t] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
        if (EF) re[g][t] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rsE, off, 0, 0));
      }
    }
  };
  // column operand of tile q (segment sg_i): its image (hi and lo fragments
  // in LDS order, 2 TS x 16 bytes per 64 columns; rank b's at img_bs bytes
  // from rank 0's) copied HBM -> LDS with no registers; each wave copies CPW
  // consecutive 1-KiB pieces (a tile past the run, q >= Q, copies zeros from
  // past the range: no fetch)
  auto copy_c = [&](int q, int sg_i, uint4 *ring) {
    int b, rb, j0;
    coord(q < Q ? q : Q - 1, b, rb, j0);
    const char *img = static_cast<const char *>(sg_i ? p.col_img2 : p.col_img) + (int64_t)b * (sg_i ? p.img_bs2 : p.img_bs);
    const __amdgpu_buffer_rsrc_t rsI = __builtin_amdgcn_make_buffer_rsrc(
        (void *)img, (short)0, (int)((int64_t)(N32 / 64) * 2 * TS * 16), 0x00020000);
    const uint32_t src = q < Q ? (uint32_t)(j0 / 64) * (uint32_t)(2 * TS * 16) + (uint32_t)(wave * CPW * 1024 + lane * 16)
                               : 0x80000000u;
#pragma unroll
    for (int i = 0; i < CPW; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsI, (GIFT_LDS void *)(ring + (wave * CPW + i) * 64), 16,
                                               (int)(src + (uint32_t)i * 1024u), 0, 0, 0);
  };
  // row operand (segment sg_i) of the wave's rows 16 g .. + 15 of row
  // block rb of rank b, loaded, then split into chunks sg_i KC .. of rh /
  // rl (two segments: one 16-row group's loads at a time, which keeps the
  // split fragments of both segments and one group in flight under 256
  // registers)
  constexpr int RWG = NSEG == 2 ? 1 : 2;
  float4 rw[RWG][KC][2];
  uint4 rh[2][NCH], rl[2][NCH];
  auto load_r = [&](int b, int rb, int sg_i, int g) {
    const LUSeg &sq = p.seg[sg_i];
    const int r = rb * kUpdRows + wave * 32 + 16 * g + fr;
    const bool ok = r < M32;
    const float *q = sq.row + (int64_t)b * sq.row_bs + (int64_t)(ok ? r : 0) * sq.row_ld + 4 * fg;
#pragma unroll
    for (int ch = 0; ch < KC; ++ch) {
      rw[g % RWG][ch][0] = ld4_if(ok, q + 32 * ch);
      rw[g % RWG][ch][1] = ld4_if(ok, q + 32 * ch + 16);
    }
  };
  auto split_r = [&](int sg_i, int g) {
#pragma unroll
    for (int ch = 0; ch < KC; ++ch)
      split8(rw[g % RWG][ch][0], rw[g % RWG][ch][1], rh[g][sg_i * KC + ch], rl[g][sg_i * KC + ch]);
  };
  // the row operand of row block rb of rank b, both groups of every segment
  auto reload_r = [&](int b, int rb) {
    if (NSEG == 1) {
      load_r(b, rb, 0, 0);
      load_r(b, rb, 0, 1);
      split_r(0, 0);
      split_r(0, 1);
    } else {
#pragma unroll
      for (int s2 = 0; s2 < NSEG; ++s2)
#pragma unroll
        for (int g = 0; g < 2; ++g) {
          load_r(b, rb, s2, g);
          split_r(s2, g);
        }
    }
  };
  // QUANT: raw sub-slot `lane` of tile q's block
  auto load_raw = [&](int q) -> uint32_t {
    int b, rb, j0;
    coord(q, b, rb, j0);
    const int i0 = rb * kUpdRows + wave * 32;   // a wave past M reads the last block row (not used)
    const int gb = b * nblk + ((i0 < M32 ? i0 : M32 - 1) / br) * (int)p.nbc + j0 / bc;
    return p.raw[gb * kAmaxSlots + lane];
  };

  int cur_b, cur_rb;
  {
    int j0;
    coord(0, cur_b, cur_rb, j0);
  }
  WTile dA, dB, rA, rB;
  uint32_t rawA = 0u, rawB = 0u;
  if (NSEG == 2) {   // segment 1's rows and segment 0's first group split ahead
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      load_r(cur_b, cur_rb, 1, g);
      split_r(1, g);
    }
    load_r(cur_b, cur_rb, 0, 0);
    split_r(0, 0);
    load_r(cur_b, cur_rb, 0, 1);
  } else {
    load_r(cur_b, cur_rb, 0, 0);
    load_r(cur_b, cur_rb, 0, 1);
  }
  copy_c(0, 0, ring0);
  load_w(0, dA, rA);
  if (DEEP) load_w(1, dB, rB);
  if (EPI == EPI_QUANT) {
    rawA = load_raw(0);
    if (DEEP) rawB = load_raw(1);
  }
  __builtin_amdgcn_sched_barrier(0);   // every prologue load ahead of the first wait
  if (NSEG == 1) split_r(0, 0);
  split_r(0, 1);
  // this wave's copies into ring0 done (the 16 W and 0 / 2 raw loads issued
  // after them may still be in flight), then everyone's
  wait_vm<(DEEP ? 2 : 1) * ((EF ? 16 : 8) + (EPI == EPI_QUANT ? 1 : 0))>();
  __syncthreads();

  uint32_t run_max = 0u;
  int run_blk = -1;
  int q_blk = -1;
  float q_inv = 0.f, q_s = 0.f;
  // two segments: one segment's products issued with the LDS reads of the
  // next 16 columns one step ahead of their products (two reads, then six
  // products), so that two steps' fragments at most are held in registers
  auto pipe_one_ahead = [&]() {
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
#pragma unroll
    for (int i = 1; i < 4 * KC; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 6, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 6, 0);
  };
  // tile q (h = q & 1, a constant at each call)
  auto tile = [&](int q, const int h, WTile &cur, WTile &curR, uint32_t &raw) {
    int b, rb, j0;
    coord(q, b, rb, j0);
    uint4 *const rd = NSEG == 2 || h == 0 ? ring0 : ring1;
    // one segment: the next tile's column operand into the other half (all
    // waves left it at the end of the previous tile); two: this tile's
    // segment 1 into ring1
    if (NSEG == 1) copy_c(q + 1, 0, h ? ring0 : ring1);
    else copy_c(q, 1, ring1);
    __builtin_amdgcn_sched_barrier(0);
    if (h == 0 && (b != cur_b || rb != cur_rb)) {   // a new row block (workgroup-uniform)
      cur_b = b;
      cur_rb = rb;
      reload_r(b, rb);
    }
    const int i0 = rb * kUpdRows + wave * 32;
    floatx4 acc[2][4];
#pragma unroll
    for (int g = 0; g < 2; ++g)
#pragma unroll
      for (int t = 0; t < 4; ++t) acc[g][t] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ch = 0; ch < KC; ++ch)
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int e = ch * 256 + lds_slot(16 * t + fr, fg);
        const uint4 ah = rd[e], al = rd[TS + e];
#pragma unroll
        for (int g = 0; g < 2; ++g) acc[g][t] = mfma3(ah, al, rh[g][ch], rl[g][ch], acc[g][t]);
      }
    if (NSEG == 2) {
      // this wave's copies of segment 1 done (nothing issued after them),
      // then everyone's; everyone is done with ring0: the next tile's
      // segment 0 goes there under segment 1's products
      wait_vm<0>();
      __syncthreads();
      copy_c(q + 1, 0, ring0);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int ch = KC; ch < NCH; ++ch)
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int e = (ch - KC) * 256 + lds_slot(16 * t + fr, fg);
          const uint4 ah = ring1[e], al = ring1[TS + e];
#pragma unroll
          for (int g = 0; g < 2; ++g) acc[g][t] = mfma3(ah, al, rh[g][ch], rl[g][ch], acc[g][t]);
        }
    }
    if (i0 < M32) {
      bool rv[2];
#pragma unroll
      for (int g = 0; g < 2; ++g) rv[g] = i0 + 16 * g + fr < M32;
      float w[2][4][4];
#pragma unroll
      for (int g = 0; g < 2; ++g)
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          w[g][t][0] = cur[g][t].x + acc[g][t][0];
          w[g][t][1] = cur[g][t].y + acc[g][t][1];
          w[g][t][2] = cur[g][t].z + acc[g][t][2];
          w[g][t][3] = cur[g][t].w + acc[g][t][3];
          if (EF) {
            w[g][t][0] += curR[g][t].x;
            w[g][t][1] += curR[g][t].y;
            w[g][t][2] += curR[g][t].z;
            w[g][t][3] += curR[g][t].w;
          }
        }
      const int bi = i0 / br, bj = j0 / bc;
      const int gb = b * nblk + bi * (int)p.nbc + bj;
      if (WT) {   // W~ of the tile for the streaming quantize pass
#pragma unroll
        for (int g = 0; g < 2; ++g)
          if (rv[g]) {
            float *dst = p.transformed + (int64_t)b * MN + (int64_t)(i0 + 16 * g + fr) * N32 + j0 + 4 * fg;
#pragma unroll
            for (int t = 0; t < 4; ++t)
              st_u128_untracked(dst + 16 * t, make_uint4(__float_as_uint(w[g][t][0]), __float_as_uint(w[g][t][1]),
                                                         __float_as_uint(w[g][t][2]), __float_as_uint(w[g][t][3])));
          }
      }
      if (EPI == EPI_AMAX) {
        uint32_t m = 0u;
#pragma unroll
        for (int g = 0; g < 2; ++g)
          if (rv[g]) {
#pragma unroll
            for (int t = 0; t < 4; ++t)
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const uint32_t a = __float_as_uint(w[g][t][e]) & 0x7fffffffu;
                m = a > m ? a : m;
              }
          }
        m = wave_max_u32(m);
        if (gb != run_blk) {
          if (run_blk >= 0 && lane == 0 && run_max) atomicMax(&p.amax[run_blk * kAmaxSlots + slot], run_max);
          run_blk = gb;
          run_max = 0u;
        }
        run_max = m > run_max ? m : run_max;
      } else {
        if (gb != q_blk) {
          const float a = __uint_as_float(wave_max_u32(raw));
          q_inv = e4m3_multiplier(a);
          q_s = e4m3_scale(a);
          q_blk = gb;
          if (lane == 0 && i0 == bi * br && j0 == bj * bc)
            st_u32_untracked(p.scales + gb, __float_as_uint(e4m3_scale(a)));
        }
#pragma unroll
        for (int g = 0; g < 2; ++g)
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const uint32_t packed = e4m3_encode4(w[g][t][0] * q_inv, w[g][t][1] * q_inv, w[g][t][2] * q_inv,
                                                 w[g][t][3] * q_inv);
            cstage[wave][(16 * g + fr) * 32 + 16 * h + 4 * t + fg] = packed;
            if (EF && rv[g]) {   // R = W~ - its dequantized code
              float qv[4];
              e4m3_decode4(packed, qv);
              st_u128_untracked(p.ef + (int64_t)b * MN + (int64_t)(i0 + 16 * g + fr) * N32 + j0 + 16 * t + 4 * fg,
                                make_uint4(__float_as_uint(w[g][t][0] - qv[0] * q_s),
                                           __float_as_uint(w[g][t][1] - qv[1] * q_s),
                                           __float_as_uint(w[g][t][2] - qv[2] * q_s),
                                           __float_as_uint(w[g][t][3] - qv[3] * q_s)));
            }
          }
        if (h == 1) {
          // the pair's codes, whole 128-byte lines; the wave reads back only
          // what its own lanes wrote, and one wave's LDS accesses complete in
          // order: wavefront-scope fences keep the compiler from reordering
          // them without waiting for this wave's loads in flight
          __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
          __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
          // 16-byte chunk lane + 64 h: row lane / 8 + 8 h, chunk lane % 8
          const int row0 = lane >> 3, qt = lane & 7;
          const uint4 *src = reinterpret_cast<const uint4 *>(&cstage[wave][row0 * 32 + 4 * qt]);
          uint8_t *cb = p.codes + (int64_t)b * MN + (int64_t)(i0 + row0) * N32 + (j0 - 64 + 16 * qt);
#pragma unroll
          for (int h = 0; h < 4; ++h) {
            const uint4 v = src[64 * h];
            if (i0 + row0 + 8 * h < M32) st_u128_untracked(cb + (int64_t)(8 * h) * N32, v);
          }
        }
      }
    }
    // W of the tile after next (past the run: zeros, unfetched, loaded all
    // the same so that every wait stays exact)
    const int qn = DEEP ? q + 2 : q + 1;
    __builtin_amdgcn_sched_barrier(0);
    load_w(qn, cur, curR);
    if (EPI == EPI_QUANT) raw = load_raw(qn < Q ? qn : Q - 1);
    // this wave's copies of the next tile done (only the 8 W (+ 8 residual)
    // and 0 / 1 raw loads above may still be in flight: loads complete in
    // order), then everyone's
    wait_vm<(EF ? 16 : 8) + (EPI == EPI_QUANT ? 1 : 0)>();
    __syncthreads();
  };
  for (int q = 0; q < Q; q += 2) {
    tile(q, 0, dA, rA, rawA);
    if (DEEP) tile(q + 1, 1, dB, rB, rawB);
    else tile(q + 1, 1, dA, rA, rawA);
  }
  if (EPI == EPI_AMAX && run_blk >= 0 && lane == 0 && run_max)
    atomicMax(&p.amax[run_blk * kAmaxSlots + slot], run_max);
}

template <int EPI, int KC, bool EF = false, int NSEG = 1, bool WT = false>
__global__ __launch_bounds__(kUpdThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void lr_sweep_kernel(
    const LUArgs p) {
  lr_sweep_body<EPI, KC, EF, NSEG, WT>(p);
}

// ---------------------------------------------------------------------------
// Transposed projection Q^T = W^T U (the output side's U_G^T W of eq.
// design_full_transform, stored n x r) with split-bf16 products: out[j][k] =
// sum_i W[i][j] U[i][k] for k < r = 64 KGW, U given as U^T ([r][K] rows).
// The contraction runs over W's rows, which no register layout reads
// contiguously, so W goes through LDS: each 32-row stage of a 64-column
// tile is copied HBM -> LDS with no registers (four-stage ring, three
// stages in flight), the 16-column chunks of row i at chunk position
// g ^ ((i >> 2) & 3), and each lane reads its eight rows of one column with
// 32-bit LDS reads (conflict-free under that swizzle) and splits them into
// the matrix-core operand.  A workgroup's four waves split r (16 KGW
// columns each) and share the 64 columns of W; U^T comes straight from L2
// (every workgroup reads all of it).  The products are those of the bf16
// hi / lo split of both operands (hi hi + hi lo + lo hi), accumulated in
// float32 over the stages in order: deterministic.  Split-K: workgroup z of
// a column tile takes rows [z rps, (z + 1) rps) and writes partial z.
// ---------------------------------------------------------------------------

constexpr int kPtStage = 32;   // rows of W per stage (four-slot LDS ring)

struct PTArgs {
  const float *W = nullptr;    // [batch][K][M] (M contiguous)
  int64_t wbs = 0;             // floats between ranks' W
  int K = 0, M = 0;            // rows of W (contraction), columns of W (output rows)
  const float *Ut = nullptr;   // [r][K], shared by the batch
  float *C = nullptr;          // [batch][ks][M][r]
  int64_t cbs = 0;             // floats between partials (M r)
  int ks = 1, rps = 0;         // partials, rows per partial (a multiple of 32)
};

template <int KGW>
__global__ __launch_bounds__(256) void lr_projT_kernel(const PTArgs p) {
  constexpr int R = 64 * KGW;
  // the four ring slots as separate arrays, so that the compiler's wait
  // analysis tells the copies into one slot from reads of another
  __shared__ __attribute__((aligned(1024))) float ring0[kPtStage * 64], ring1[kPtStage * 64],
      ring2[kPtStage * 64], ring3[kPtStage * 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int fr = lane & 15, fg = lane >> 4;
  const int tiles_j = p.M / 64;
  const int lin = (int)blockIdx.x;
  const int tj = lin % tiles_j;
  const int bz = lin / tiles_j;
  const int z = bz % p.ks, b = bz / p.ks;
  const int j0 = 64 * tj;
  const int ibeg = z * p.rps;
  const int iend = ibeg + p.rps < p.K ? ibeg + p.rps : p.K;
  // stages of the part, padded to whole rounds of the four-slot ring (rows
  // at or past iend read zeros and add nothing)
  const int nst = (iend - ibeg + 4 * kPtStage - 1) / (4 * kPtStage) * 4;   // >= 4 (launcher: part non-empty)
  const int kb = wave * 16 * KGW;

  // W stage s -> ring slot s % 4: piece 2 wave + h is LDS rows 4 (2 wave + h)
  // .. + 3; lane l lands at row + (l >> 4), chunk position (l & 15) >> 2,
  // float4 l & 3, so it fetches W[row][16 (pos ^ ((row >> 2) & 3)) + 4 (l & 3)]
  const __amdgpu_buffer_rsrc_t rsW = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(p.W + (int64_t)b * p.wbs), (short)0, (int)((int64_t)p.K * p.M * 4), 0x00020000);
  int wrow[2], wcol[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    wrow[h] = 4 * (2 * wave + h) + (lane >> 4);
    wcol[h] = j0 + 16 * (((lane & 15) >> 2) ^ ((wrow[h] >> 2) & 3)) + 4 * (lane & 3);
  }
  auto dma = [&](int s, float *dst) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int i = ibeg + kPtStage * s + wrow[h];
      const uint32_t off = i < iend ? ((uint32_t)i * (uint32_t)p.M + (uint32_t)wcol[h]) * 4u : 0x80000000u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsW, (GIFT_LDS void *)(dst + (2 * wave + h) * 256), 16, (int)off, 0,
                                               0, 0);
    }
  };
  // U^T rows kb + 16 g + fr, columns i0 + 4 fg and i0 + 16 + 4 fg of stage s
  // (the k order of the matrix-core operand used throughout this file)
  const __amdgpu_buffer_rsrc_t rsU =
      __builtin_amdgcn_make_buffer_rsrc((void *)p.Ut, (short)0, (int)((int64_t)R * p.K * 4), 0x00020000);
  typedef float4 BSet[KGW][2];
  auto load_b = [&](int s, BSet &bs) {
    const int i = ibeg + kPtStage * s + 4 * fg;
#pragma unroll
    for (int g = 0; g < KGW; ++g)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int ii = i + 16 * h;
        const uint32_t off =
            ii < iend ? ((uint32_t)(kb + 16 * g + fr) * (uint32_t)p.K + (uint32_t)ii) * 4u : 0x80000000u;
        bs[g][h] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rsU, (int)off, 0, 0));
      }
  };

  floatx4 acc[4][KGW];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int g = 0; g < KGW; ++g) acc[a][g] = floatx4{0.f, 0.f, 0.f, 0.f};

  BSet bA, bB;
  // prologue: U^T of stage 0, then W of stages 0 .. 2; the wait for stage
  // 0's U^T covers nothing after it
  load_b(0, bA);
  dma(0, ring0);
  dma(1, ring1);
  dma(2, ring2);
  copies_barrier<4>();   // stage 0 landed everywhere (stages 1, 2 may be in flight)

  // stage s: U^T of stage s + 1 (into the other set), then W of stage s + 3
  // into the slot read at stage s - 1 (all waves left it: barrier), then
  // the products of stage s.  Completing U^T(s + 1) (waited for at stage
  // s + 1) implies W(s + 2) landed (issued before it), so the W copies run
  // two to three stages ahead of their use.
  auto stage = [&](int s, const float *src, float *next3, BSet &cur, BSet &nxt) {
    load_b(s + 1, nxt);
    dma(s + 3, next3);
    __builtin_amdgcn_sched_barrier(0);   // both issued ahead of this stage's products
    uint4 bh[KGW], bl[KGW];
#pragma unroll
    for (int g = 0; g < KGW; ++g) split8(cur[g][0], cur[g][1], bh[g], bl[g]);
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      // column 16 a + fr, rows 4 fg .. + 3 and 16 + 4 fg .. + 3 (both with
      // (row >> 2) & 3 = fg: chunk position a ^ fg)
      const float *c = src + 16 * (a ^ fg) + fr;
      float4 lo, hi;
      lo.x = c[(4 * fg + 0) * 64];
      lo.y = c[(4 * fg + 1) * 64];
      lo.z = c[(4 * fg + 2) * 64];
      lo.w = c[(4 * fg + 3) * 64];
      hi.x = c[(16 + 4 * fg + 0) * 64];
      hi.y = c[(16 + 4 * fg + 1) * 64];
      hi.z = c[(16 + 4 * fg + 2) * 64];
      hi.w = c[(16 + 4 * fg + 3) * 64];
      uint4 ah, al;
      split8(lo, hi, ah, al);
#pragma unroll
      for (int g = 0; g < KGW; ++g) acc[a][g] = mfma3(ah, al, bh[g], bl[g], acc[a][g]);
    }
    // this wave's W of stage s + 1 landed (only W(s + 2), U^T(s + 1) and
    // W(s + 3) may be in flight: 2 + 2 KGW + 2), then everyone's; everyone
    // is done with slot s % 4
    copies_barrier<4 + 2 * KGW>();
  };
  for (int s = 0; s < nst; s += 4) {
    stage(s, ring0, ring3, bA, bB);
    stage(s + 1, ring1, ring0, bB, bA);
    stage(s + 2, ring2, ring1, bA, bB);
    stage(s + 3, ring3, ring2, bB, bA);
  }

  // lane holds out[j0 + 16 a + 4 fg + e][kb + 16 g + fr]
  float *out = p.C + ((int64_t)b * p.ks + z) * p.cbs;
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int g = 0; g < KGW; ++g)
#pragma unroll
      for (int e = 0; e < 4; ++e) out[(int64_t)(j0 + 16 * a + 4 * fg + e) * R + kb + 16 * g + fr] = acc[a][g][e];
}

bool al16(const void *q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; }

}  // namespace

int lr_proj_parts(int64_t M, int64_t K, int32_t batch) {
  // at least two workgroups per CU, each part at least two stages deep, and
  // at most four partials: every partial is written, read back and summed,
  // so more of them than that costs more HBM traffic than the extra
  // parallelism saves (measured on the MLP shapes: 2 instead of 4 partials
  // for the 5632 x 1024 gate + up bucket, 1408 -> 704 workgroups, makes the
  // projection 7 % faster and the concurrent step 1.5 %). Launches of 128
  // row tiles or more stop at two partials (one workgroup per CU already):
  // on the Llama-600M o and down buckets (192 tiles of 16 ranks) 2 instead
  // of 4 made the projection about 2 % slower alone and the four-stream
  // codec step 37.38-37.50 -> 37.29-37.33 ms over three alternating runs
  // (half the partials' traffic; the step is bound by its HBM bytes)
  const int64_t tiles = (M + kProjRows - 1) / kProjRows * batch;
  const int max_parts = tiles >= 128 ? 2 : 4;
  int parts = 1;
  while (parts < max_parts && tiles * parts < 512 && K / (2 * parts) >= 2 * kProjStage) parts *= 2;
  return parts;
}

// The projection kernel takes its 16-row strips from the operand with the
// long side: rows of A (out[i][c] = C[i][c], split-K partials allowed) or,
// for a short output (M <= 128 rows), rows of B with the result stored
// transposed into C[c][j].
static bool lr_strip_is_b(const TileJob &j) { return j.M <= 128 && j.N > j.M; }

bool lr_proj_eligible(const TileJob &j) {
  const Segment &g = j.seg[0];
  const bool tr = lr_strip_is_b(j);
  const int64_t C = tr ? j.M : j.N;
  const Operand &xs = tr ? g.b : g.a, &ys = tr ? g.a : g.b;
  if (!(j.split3 && j.nseg == 1 && j.amax == nullptr && j.alpha == 1.f &&
        (C == 16 || C == 32 || C == 64 || C == 128) && g.a.kmajor && g.b.kmajor && g.K % 4 == 0 &&
        xs.ld == g.K && ys.ld == g.K && xs.bs % 4 == 0 && ys.bs % 4 == 0 && al16(xs.ptr) && al16(ys.ptr) &&
        !job_has_tabs(j)))
    return false;
  // an addend and column scales: whole, untransposed, one partial
  if ((j.D || j.colscale) &&
      (tr || j.ksplit > 1 || j.beta != 1.f || (j.D && (!al16(j.D) || j.ldd != C || j.dbs != j.M * C)) ||
       (j.colscale && !al16(j.colscale))))
    return false;
  if (tr) return j.ksplit <= 1;
  return al16(j.C) && j.ldc == C && j.cbs == j.M * C && (j.ksplit <= 1 || ys.bs == 0);
}

gift_status launch_lr_proj(gift_ctx *ctx, const TileJob &j) {
  const bool tr = lr_strip_is_b(j);
  const Operand &xs = tr ? j.seg[0].b : j.seg[0].a, &ys = tr ? j.seg[0].a : j.seg[0].b;
  const int64_t C = tr ? j.M : j.N;
  LPArgs a{};
  a.X = xs.ptr;
  a.x_bs = xs.bs;
  a.Y = ys.ptr;
  a.y_bs = ys.bs;
  a.M = tr ? j.N : j.M;
  a.K = j.seg[0].K;
  a.out = j.C;
  a.parts = j.ksplit > 1 ? j.ksplit : 1;
  a.kper = ((a.K + a.parts - 1) / a.parts + kProjStage - 1) / kProjStage * kProjStage;
  a.out_t = tr ? 1 : 0;
  a.out_ld = j.ldc;
  a.out_bs = j.cbs;
  a.D = j.D;
  a.d_bs = j.dbs;
  a.colscale = j.colscale;
  ProfileScope prof(ctx, j.kernel_family);
  const dim3 grid((unsigned)((a.M + kProjRows - 1) / kProjRows), (unsigned)a.parts, (unsigned)j.batch);
  switch (C) {
    case 16: hipLaunchKernelGGL(lr_proj_kernel<1>, grid, dim3(kProjThreads), 0, ctx->stream, a); break;
    case 32: hipLaunchKernelGGL(lr_proj_kernel<2>, grid, dim3(kProjThreads), 0, ctx->stream, a); break;
    case 64: hipLaunchKernelGGL(lr_proj_kernel<4>, grid, dim3(kProjThreads), 0, ctx->stream, a); break;
    default: hipLaunchKernelGGL(lr_proj_kernel<8>, grid, dim3(kProjThreads), 0, ctx->stream, a); break;
  }
  return check_launch("lr_proj_kernel");
}

// rows per part of a K-row contraction split ks ways (whole 128-row rounds)
int64_t lr_projT_rows(int64_t K, int ks) {
  return ((K + ks - 1) / ks + 4 * kPtStage - 1) / (4 * kPtStage) * (4 * kPtStage);
}

int lr_projT_parts(int64_t M, int64_t K, int64_t r, int32_t batch) {
  if (!(r == 64 || r == 128) || M <= 0 || M % 64 != 0 || K <= 0 || K % 4 != 0 || K * M >= (1LL << 29) ||
      batch < 1 || (M / 64) * (int64_t)batch >= (1LL << 30))
    return 0;
  // split the rows while the launch holds under 512 workgroups and each
  // part keeps at least 128 rows; parts of whole rounds of the four-stage
  // ring (128 rows)
  const int64_t tiles = M / 64 * batch;
  int ks = 1;
  while (ks < 16 && tiles * ks < 512 && K / (2 * ks) >= 128) ks *= 2;
  const int64_t rps = lr_projT_rows(K, ks);
  return (int)((K + rps - 1) / rps);
}

bool lr_projT_eligible(const TileJob &j) {
  if (j.nseg != 1 || j.split3 == false || j.D != nullptr || j.colscale != nullptr || j.alpha != 1.f ||
      j.beta != 0.f || j.amax || j.codes || j.mx_codes || j.decode_tab || job_has_tabs(j))
    return false;
  const Segment &g = j.seg[0];
  const int parts = lr_projT_parts(j.M, g.K, j.N, j.batch);
  return parts > 0 && parts == j.ksplit && !g.a.kmajor && g.a.ld == j.M && g.a.bs == g.K * j.M && g.b.kmajor &&
         g.b.ld == g.K && g.b.bs == 0 && g.b.parts <= 1 && g.a.parts <= 1 && j.ldc == j.N && j.cbs == j.M * j.N &&
         al16(g.a.ptr) && al16(g.b.ptr) && al16(j.C);
}

gift_status launch_lr_projT(gift_ctx *ctx, const TileJob &j) {
  if (!lr_projT_eligible(j)) return GIFT_EUNSUPPORTED;
  const Segment &g = j.seg[0];
  PTArgs a{};
  a.W = g.a.ptr;
  a.wbs = g.a.bs;
  a.K = (int)g.K;
  a.M = (int)j.M;
  a.Ut = g.b.ptr;
  a.C = j.C;
  a.cbs = j.cbs;
  a.ks = j.ksplit;
  a.rps = (int)lr_projT_rows(g.K, j.ksplit);
  // every part non-empty (lr_projT_parts)
  if ((int64_t)(a.ks - 1) * a.rps >= g.K) return GIFT_EUNSUPPORTED;
  const int64_t wgs = j.M / 64 * (int64_t)j.batch * j.ksplit;
  ProfileScope prof(ctx, j.kernel_family);
  if (j.N == 64)
    hipLaunchKernelGGL(lr_projT_kernel<1>, dim3((unsigned)wgs), dim3(256), 0, ctx->stream, a);
  else
    hipLaunchKernelGGL(lr_projT_kernel<2>, dim3((unsigned)wgs), dim3(256), 0, ctx->stream, a);
  return check_launch("lr_projT_kernel");
}

size_t lr_col_image_bytes(int64_t N, int K) {
  if (N <= 0 || N % 128 != 0 || !(K == 64 || K == 96 || K == 128)) return 0;
  return (size_t)N * (size_t)K * 4;   // hi + lo bf16 per element
}

gift_status launch_lr_col_image(gift_ctx *ctx, const float *col, int64_t ld, int64_t N, int K, void *img,
                                int32_t count, int64_t col_bs) {
  if (lr_col_image_bytes(N, K) == 0 || count < 1) return GIFT_ESHAPE;
  const int nch = K / 32;
  const int64_t entries = N / 64 * nch * 256;
  const int64_t blocks = std::min<int64_t>((entries * count + 255) / 256, 2048);
  ProfileScope prof(ctx, GIFT_KERNEL_PROJECT);
  hipLaunchKernelGGL(lr_col_image_kernel, dim3((unsigned)blocks), dim3(256), 0, ctx->stream, col, ld, col_bs, entries,
                     (int64_t)count, nch, static_cast<uint4 *>(img));
  return check_launch("lr_col_image_kernel");
}

gift_status launch_lr_psum(gift_ctx *ctx, const float *partials, float *out, int parts, int64_t per_rank,
                           int32_t batch, int kernel_family) {
  const int64_t total = per_rank * batch;
  const int64_t blocks = std::min<int64_t>((total / 4 + 255) / 256, 4096);
  ProfileScope prof(ctx, kernel_family);
  hipLaunchKernelGGL(lr_psum_kernel, dim3((unsigned)std::max<int64_t>(blocks, 1)), dim3(256), 0, ctx->stream,
                     partials, out, parts, per_rank, total);
  return check_launch("lr_psum_kernel");
}

bool lr_quant_reads_raw(const TileJob &j) {
  // every 32 x 64 wave tile inside one scale block
  const int64_t br = j.geom.br > 0 ? j.geom.br : j.M, bc = j.geom.bc > 0 ? j.geom.bc : j.N;
  return (br % 32 == 0 || br >= j.M) && (bc % 64 == 0 || bc >= j.N) && kAmaxSlots == 64;
}

bool lr_update_eligible(const TileJob &j) {
  const bool mx = j.mx_codes != nullptr;
  if (!j.split3 || (j.amax == nullptr && !mx) || j.nseg < 1 || j.nseg > 2 || j.N % 4 != 0) return false;
  if (mx && (j.N % 32 != 0 || j.codes != nullptr || (reinterpret_cast<uintptr_t>(j.mx_codes) & 1))) return false;
  if (j.M * j.N >= (1LL << 29)) return false;   // one rank's slice within a 32-bit buffer range
  const int64_t K = j.seg[0].K;
  if (K <= 0 || K > 128 || K % 4 != 0) return false;
  for (int s = 0; s < j.nseg; ++s) {
    const Segment &g = j.seg[s];
    if (!g.a.kmajor || !g.b.kmajor || g.K != K) return false;
    if (g.a.ld % 4 || g.b.ld % 4 || g.a.bs % 4 || g.b.bs % 4) return false;
    if (!al16(g.a.ptr) || !al16(g.b.ptr)) return false;
  }
  if (!al16(j.D) || j.ldd != j.N || j.dbs != j.M * j.N) return false;
  if ((j.transformed && !al16(j.transformed)) || (j.ef && !al16(j.ef)) ||
      (j.codes && (reinterpret_cast<uintptr_t>(j.codes) & 3)))
    return false;
  return true;
}

gift_status launch_lr_update(gift_ctx *ctx, const TileJob &j) {
  LUArgs a{};
  for (int s = 0; s < j.nseg; ++s) {
    a.seg[s].row = j.seg[s].a.ptr;
    a.seg[s].row_ld = j.seg[s].a.ld;
    a.seg[s].row_bs = j.seg[s].a.bs;
    a.seg[s].row_parts = j.seg[s].a.parts;
    a.seg[s].col = j.seg[s].b.ptr;
    a.seg[s].col_ld = j.seg[s].b.ld;
    a.seg[s].col_bs = j.seg[s].b.bs;
    a.seg[s].K = (int)j.seg[s].K;
  }
  a.M = j.M;
  a.N = j.N;
  a.D = j.D;
  a.amax = j.amax;
  a.codes = j.codes;
  a.hits = j.codes ? j.hits : nullptr;
  a.transformed = j.transformed;
  a.ef = j.ef;
  a.br = j.geom.br > 0 ? j.geom.br : j.M;
  a.bc = j.geom.bc > 0 ? j.geom.bc : j.N;
  a.nbr = j.geom.nbr;
  a.nbc = j.geom.nbc;
  a.codes_wide = j.codes && j.N % 16 == 0 && al16(j.codes) ? 1 : 0;
  a.raw = j.codes && j.from_raw ? j.amax : nullptr;
  a.scales = j.scales;
  a.clear = a.raw ? j.clear : nullptr;
  a.clear_words = a.raw ? j.clear_words : 0;
  a.shared = j.shared ? 1 : 0;
  a.batch = j.batch;
  a.mx_codes = j.mx_codes;
  a.mx_scales = j.mx_scales;
  ProfileScope prof(ctx, j.kernel_family);
  const int64_t cols = 64 * upd_tiles(j.nseg * (int)((j.seg[0].K + 31) / 32));
  const dim3 grid((unsigned)((j.N + cols - 1) / cols), (unsigned)((j.M + kUpdRows - 1) / kUpdRows),
                  (unsigned)j.batch);
  const bool quant = j.codes != nullptr;
  const bool ef = j.ef != nullptr;
  const int kc = (int)((j.seg[0].K + 31) / 32);
  // every wave tile inside one scale block, no optional W~ output, and for
  // QUANT the raw block maxima and whole column ranges: the variant whose
  // tile loop has no branch between its waits
  const bool full = lr_quant_reads_raw(j) && j.transformed == nullptr &&
                    (!quant || (a.raw != nullptr && a.codes_wide && j.N % cols == 0));
  // the sweep variant: whole 128-column units, per-rank scales, every wave
  // tile inside one block, no hit counts, each segment's column operand as
  // its LDS image; one segment (the input side alone, a shared column
  // operand, with or without the residual) or two (both sides: rank-2r
  // update, no residual) of one rank each, K = 64, 96 or 128
  const int64_t sw_units = j.batch * ((j.M + kUpdRows - 1) / kUpdRows) * (j.N / 128);
  const int64_t K0 = j.seg[0].K;
  const bool seg_ok =
      j.nseg == 1 ? j.col_img != nullptr && j.seg[0].a.parts == 1 && j.seg[0].b.bs == 0 && j.img_bs == 0
                  : j.nseg == 2 && !ef && j.col_img != nullptr && j.col_img2 != nullptr && j.seg[0].a.parts == 1 &&
                        j.seg[1].a.parts == 1 && j.seg[1].K == K0 && j.img_bs >= 0 && j.img_bs2 >= 0;
  // (the two-segment AMAX pass at rank 96 or 128 may also store W~ for a
  // streaming quantize pass: sweep_store)
  const bool wt_store = j.transformed != nullptr && j.sweep_store && !quant && j.nseg == 2 && (K0 == 96 || K0 == 128) &&
                        al16(j.transformed);
  const bool full_sw = full || (wt_store && lr_quant_reads_raw(j));
  const bool sweep = full_sw && seg_ok && !j.mx_codes && !(quant && j.hits) && (K0 == 64 || K0 == 96 || K0 == 128) &&
                     j.N % 128 == 0 && !j.shared && sw_units > 0 && sw_units < (1LL << 30) &&
                     (int64_t)j.batch * j.geom.nbr * j.geom.nbc * kAmaxSlots < (1LL << 31);
  if (sweep) {
    // runs of four units (eight 64-column tiles) once the launch fills four
    // rounds of resident workgroups (two per CU), shorter runs below.
    // Measured on the Llama-600M buckets in the four-stream step: runs of
    // 3-4 units 38.8-39.6 ms per codec step, 5-6 units 43-45 ms, runs sized
    // for one or two rounds 46-47 ms (the same kernels in isolation differ
    // by under 5 %)
    const int64_t upw = sw_units >= 4 * 512 ? 4 : std::max<int64_t>(1, sw_units / 512);
    a.upw = (int)upw;
    a.col_img = j.col_img;
    a.img_bs = j.img_bs;
    a.col_img2 = j.nseg == 2 ? j.col_img2 : nullptr;
    a.img_bs2 = j.nseg == 2 ? j.img_bs2 : 0;
    const dim3 sgrid((unsigned)((sw_units + upw - 1) / upw));
    auto sgo = [&](auto epi_c, auto ef_c, auto nseg_c) {
      constexpr int E = decltype(epi_c)::value;
      constexpr bool R = decltype(ef_c)::value;
      constexpr int S = decltype(nseg_c)::value;
      if constexpr (S == 2 && !R && E == EPI_AMAX) {
        if (wt_store) {
          if (K0 == 96)
            hipLaunchKernelGGL((lr_sweep_kernel<E, 3, false, 2, true>), sgrid, dim3(kUpdThreads), 0, ctx->stream, a);
          else
            hipLaunchKernelGGL((lr_sweep_kernel<E, 4, false, 2, true>), sgrid, dim3(kUpdThreads), 0, ctx->stream, a);
          return;
        }
      }
      if constexpr (S == 1 || !R) {
        switch (K0) {
          case 64: hipLaunchKernelGGL((lr_sweep_kernel<E, 2, R, S>), sgrid, dim3(kUpdThreads), 0, ctx->stream, a); break;
          case 96: hipLaunchKernelGGL((lr_sweep_kernel<E, 3, R, S>), sgrid, dim3(kUpdThreads), 0, ctx->stream, a); break;
          default: hipLaunchKernelGGL((lr_sweep_kernel<E, 4, R, S>), sgrid, dim3(kUpdThreads), 0, ctx->stream, a); break;
        }
      }
    };
    using One = std::integral_constant<int, 1>;
    using Two = std::integral_constant<int, 2>;
    if (quant) {
      if (ef) sgo(std::integral_constant<int, EPI_QUANT>{}, std::true_type{}, One{});
      else if (j.nseg == 2) sgo(std::integral_constant<int, EPI_QUANT>{}, std::false_type{}, Two{});
      else sgo(std::integral_constant<int, EPI_QUANT>{}, std::false_type{}, One{});
    } else {
      if (ef) sgo(std::integral_constant<int, EPI_AMAX>{}, std::true_type{}, One{});
      else if (j.nseg == 2) sgo(std::integral_constant<int, EPI_AMAX>{}, std::false_type{}, Two{});
      else sgo(std::integral_constant<int, EPI_AMAX>{}, std::false_type{}, One{});
    }
    return check_launch("lr_sweep_kernel");
  }
  auto go = [&](auto epi_c, auto ef_c, auto nseg_c, auto kc_c) {
    constexpr int E = decltype(epi_c)::value;
    constexpr bool EFv = decltype(ef_c)::value;
    constexpr int NS = decltype(nseg_c)::value, KCv = decltype(kc_c)::value;
    if constexpr (E == EPI_AMAX || E == EPI_QUANT) {
      if (full) {
        if constexpr (upd_two_waves(E, EFv, NS * KCv, true)) {
          hipLaunchKernelGGL((lr_update_kernel_o2<E, EFv, NS, KCv, true>), grid, dim3(kUpdThreads), 0,
                             ctx->stream, a);
          return;
        } else if constexpr (!upd_two_waves(E, EFv, NS * KCv, false)) {
          hipLaunchKernelGGL((lr_update_kernel<E, EFv, NS, KCv, true>), grid, dim3(kUpdThreads), 0,
                             ctx->stream, a);
          return;
        }
        // else: the general variant at two waves per SIMD beats the
        // branch-free one at one
      }
    }
    if constexpr (upd_two_waves(E, EFv, NS * KCv, false))
      hipLaunchKernelGGL((lr_update_kernel_o2<E, EFv, NS, KCv>), grid, dim3(kUpdThreads), 0, ctx->stream, a);
    else
      hipLaunchKernelGGL((lr_update_kernel<E, EFv, NS, KCv>), grid, dim3(kUpdThreads), 0, ctx->stream, a);
  };
  auto by_k = [&](auto epi_c, auto ef_c, auto nseg_c) {
    switch (kc) {
      case 1: go(epi_c, ef_c, nseg_c, std::integral_constant<int, 1>{}); break;
      case 2: go(epi_c, ef_c, nseg_c, std::integral_constant<int, 2>{}); break;
      case 3: go(epi_c, ef_c, nseg_c, std::integral_constant<int, 3>{}); break;
      default: go(epi_c, ef_c, nseg_c, std::integral_constant<int, 4>{}); break;
    }
  };
  auto by_seg = [&](auto epi_c, auto ef_c) {
    if (j.nseg == 1) by_k(epi_c, ef_c, std::integral_constant<int, 1>{});
    else by_k(epi_c, ef_c, std::integral_constant<int, 2>{});
  };
  using T_ = std::true_type;
  using F_ = std::false_type;
  using AMAX_ = std::integral_constant<int, EPI_AMAX>;
  using QUANT_ = std::integral_constant<int, EPI_QUANT>;
  using MX_ = std::integral_constant<int, EPI_MX>;
  if (j.mx_codes) {
    if (ef) by_seg(MX_{}, T_{});
    else by_seg(MX_{}, F_{});
  } else if (!quant) {
    if (ef) by_seg(AMAX_{}, T_{});
    else by_seg(AMAX_{}, F_{});
  } else {
    if (ef) by_seg(QUANT_{}, T_{});
    else by_seg(QUANT_{}, F_{});
  }
  return check_launch("lr_update_kernel");
}

}  // namespace gift
