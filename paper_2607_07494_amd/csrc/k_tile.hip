// Tile kernel: FP32 MFMA products fused with the codec epilogues.
//
// One workgroup (256 lanes = 4 wave64) owns a BM x BN tile of a batched
// output C[b] (M x N).  The tile accumulates up to two products A_s B_s over
// their own contraction lengths on the CDNA matrix cores
// (v_mfma_f32_16x16x4_f32, fp32 in / fp32 accumulate), staging BK = 32 wide
// K slices through LDS with a register prefetch of the next slice.  The
// epilogue then runs on the finished tile:
//
//   EPI_STORE  C = (alpha * acc + beta * D) * colscale[j]
//   EPI_AMAX   W~ = D + acc (+ R): per-block max |W~| (LDS atomics, one global
//              atomic per block and tile); optional store of W~
//   EPI_QUANT  W~ = D + acc (+ R): scale from the finished amax, E4M3 codes,
//              scale output, error-feedback residual update
//
// Without a product (nseg = 0, GEMM = false) the same epilogues are the
// Euclidean branch's amax and quantize passes over W itself.
//
// The codec epilogues implement Algorithm 1's Scale / Q / Dequantize with the
// amax rule of Sec. I (s = amax / E4M3_MAX); W~ is the transformed gradient of
// eq. design_full_transform (rank-r form: W + L R^T, see gift_api.cpp).

#include "fp8_e4m3.h"
#include "gift_internal.h"

namespace gift {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kKPad = 4;       // LDS row padding (floats)
constexpr int kMaxLocalBlocks = 256;

struct OperandP {
  const float *ptr;
  int64_t ld, bs;
  int vec;  // 16-byte loads allowed
  const float *const *tab;   // batch entry b at tab[b] (grouped decode), else ptr + b bs
};
struct SegmentP {
  OperandP a, b;
  int64_t K;
};

struct KArgs {
  SegmentP seg[2];
  int nseg;
  int ksplit;
  int64_t M, N;
  int batch;
  float *C;
  int64_t ldc, cbs;
  const float *D;
  int64_t ldd, dbs;
  float alpha, beta;
  const float *colscale;
  const float *const *colscale_tab;   // per batch entry (grouped decode), else colscale
  uint32_t *amax;
  uint8_t *codes;
  uint32_t *hits;        // QUANT: boundary-hit counters [batch][2] or null
  float *scales;
  float *transformed;
  float *ef;
  int64_t br, bc;
  int nbr, nbc;
  int shared;
  int vec_out;  // 16-byte epilogue access allowed
};

template <int ROWS, bool KMAJOR, int kBK>
struct TileLoader {
  // float4 slots of one ROWS x kBK slice
  static constexpr int kSlots = ROWS * kBK / 4;
  static constexpr int kPerThread = (kSlots + kThreads - 1) / kThreads;
  float4 r[kPerThread];

  __device__ __forceinline__ void load(const OperandP &op, int b, int64_t row0, int64_t rows,
                                       int64_t k0, int64_t K, int tid) {
    const float *base = op.tab ? op.tab[b] : op.ptr + (int64_t)b * op.bs;
#pragma unroll
    for (int s = 0; s < kPerThread; ++s) {
      const int q = tid + s * kThreads;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (q < kSlots) {
        if (KMAJOR) {
          const int row = q / (kBK / 4), kq = q % (kBK / 4);
          const int64_t gi = row0 + row, gk = k0 + 4 * kq;
          if (gi < rows) {
            const float *p = base + gi * op.ld + gk;
            if (op.vec && gk + 3 < K) {
              v = *reinterpret_cast<const float4 *>(p);
            } else {
              v.x = gk + 0 < K ? p[0] : 0.f;
              v.y = gk + 1 < K ? p[1] : 0.f;
              v.z = gk + 2 < K ? p[2] : 0.f;
              v.w = gk + 3 < K ? p[3] : 0.f;
            }
          }
        } else {
          const int kk = q / (ROWS / 4), iq = q % (ROWS / 4);
          const int64_t gk = k0 + kk, gi = row0 + 4 * iq;
          if (gk < K) {
            const float *p = base + gk * op.ld + gi;
            if (op.vec && gi + 3 < rows) {
              v = *reinterpret_cast<const float4 *>(p);
            } else {
              v.x = gi + 0 < rows ? p[0] : 0.f;
              v.y = gi + 1 < rows ? p[1] : 0.f;
              v.z = gi + 2 < rows ? p[2] : 0.f;
              v.w = gi + 3 < rows ? p[3] : 0.f;
            }
          }
        }
      }
      r[s] = v;
    }
  }

  // LDS layout: [ROWS][kBK + kKPad], contraction index contiguous.
  __device__ __forceinline__ void store(float *lds, int tid) const {
#pragma unroll
    for (int s = 0; s < kPerThread; ++s) {
      const int q = tid + s * kThreads;
      if (q < kSlots) {
        if (KMAJOR) {
          const int row = q / (kBK / 4), kq = q % (kBK / 4);
          *reinterpret_cast<float4 *>(lds + row * (kBK + kKPad) + 4 * kq) = r[s];
        } else {
          const int kk = q / (ROWS / 4), iq = q % (ROWS / 4);
          float *p = lds + (4 * iq) * (kBK + kKPad) + kk;
          p[0] = r[s].x;
          p[kBK + kKPad] = r[s].y;
          p[2 * (kBK + kKPad)] = r[s].z;
          p[3 * (kBK + kKPad)] = r[s].w;
        }
      }
    }
  }
};

template <int BM, int BN, int kBK>
struct Smem {
  static constexpr int kAB = (BM + BN) * (kBK + kKPad);
  static constexpr int kC = BM * (BN + 4);
  static constexpr int kFloats = kAB > kC ? kAB : kC;
};

__device__ __forceinline__ float block_max_abs(float a, float b) { return a > b ? a : b; }

// Local scale-block table of one output tile.
struct LocalBlocks {
  int64_t bi0, bj0;
  int nlbi, nlbj, nlb;
  __device__ __forceinline__ void init(const KArgs &p, int64_t i0, int64_t j0, int64_t i1,
                                       int64_t j1) {
    bi0 = i0 / p.br;
    bj0 = j0 / p.bc;
    nlbi = (int)((i1 - 1) / p.br - bi0 + 1);
    nlbj = (int)((j1 - 1) / p.bc - bj0 + 1);
    nlb = nlbi * nlbj;
  }
};

template <int BM, int BN, int WM, int WN, bool AK, bool BKM, bool GEMM, int EPI, int kBK>
__global__ __launch_bounds__(kThreads) void tile_kernel(const KArgs p) {
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TI = WTM / 16, TJ = WTN / 16;
  static_assert(WM * WN == 4, "four waves per workgroup");
  static_assert(TI >= 1 && TJ >= 1, "wave tile must hold whole 16x16 MFMA tiles");
  constexpr int kSmemFloats = GEMM ? Smem<BM, BN, kBK>::kFloats : 4;
  __shared__ __attribute__((aligned(16))) float smem[kSmemFloats];
  __shared__ uint32_t lds_amax[kMaxLocalBlocks];
  __shared__ float lds_inv[kMaxLocalBlocks];
  __shared__ float lds_scale[kMaxLocalBlocks];

  const int tid = threadIdx.x;
  const int zb = blockIdx.z;
  const int b = zb / p.ksplit;       // batch index
  const int ks = zb % p.ksplit;      // split-K index (STORE only)
  const int64_t i0 = (int64_t)blockIdx.y * BM;
  const int64_t j0 = (int64_t)blockIdx.x * BN;
  const int64_t i1 = i0 + BM < p.M ? i0 + BM : p.M;
  const int64_t j1 = j0 + BN < p.N ? j0 + BN : p.N;
  const int slot = (int)((blockIdx.y * gridDim.x + blockIdx.x) % kAmaxSlots);

  LocalBlocks lb;
  if (EPI != EPI_STORE) {
    lb.init(p, i0, j0, i1, j1);
    const int64_t nblk = (int64_t)p.nbr * p.nbc;
    for (int l = tid; l < lb.nlb; l += kThreads) {
      const int64_t bi = lb.bi0 + l / lb.nlbj, bj = lb.bj0 + l % lb.nlbj;
      if (EPI == EPI_AMAX) {
        if (l < kMaxLocalBlocks) lds_amax[l] = 0u;
      } else {
        const float a = __uint_as_float(p.amax[b * nblk + bi * p.nbc + bj]);
        if (l < kMaxLocalBlocks) {
          lds_inv[l] = e4m3_multiplier(a);
          lds_scale[l] = e4m3_scale(a);
        }
      }
    }
  }

  // Codec epilogue operands (W, residual) are fetched before the product so
  // their memory latency overlaps it.  Lane mapping: row tid / TPR of each
  // pass, four 4-wide column chunks interleaved across the lanes of a row.
  constexpr int TPR = BN / 16;                   // lanes per tile row
  constexpr int RPP = kThreads / TPR;            // rows per pass
  constexpr int NPASS = (BM + RPP - 1) / RPP;
  const int64_t MN = p.M * p.N;
  float4 dpre[NPASS][4], rpre[NPASS][4];
  if (EPI != EPI_STORE) {
#pragma unroll
    for (int ps = 0; ps < NPASS; ++ps) {
      const int row_l = ps * RPP + tid / TPR;
      const int64_t gi = i0 + row_l;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t gj = j0 + 4 * (tid % TPR) + (BN / 4) * v;
        float4 d = make_float4(0.f, 0.f, 0.f, 0.f), rr = d;
        if (row_l < BM && gi < p.M && gj < p.N) {
          const int64_t off = (int64_t)b * MN + gi * p.N + gj;
          if (p.vec_out && gj + 3 < p.N) {
            d = *reinterpret_cast<const float4 *>(p.D + off);
            if (p.ef) rr = *reinterpret_cast<const float4 *>(p.ef + off);
          } else {
            d.x = p.D[off];
            d.y = gj + 1 < p.N ? p.D[off + 1] : 0.f;
            d.z = gj + 2 < p.N ? p.D[off + 2] : 0.f;
            d.w = gj + 3 < p.N ? p.D[off + 3] : 0.f;
            if (p.ef) {
              rr.x = p.ef[off];
              rr.y = gj + 1 < p.N ? p.ef[off + 1] : 0.f;
              rr.z = gj + 2 < p.N ? p.ef[off + 2] : 0.f;
              rr.w = gj + 3 < p.N ? p.ef[off + 3] : 0.f;
            }
          }
        }
        dpre[ps][v] = d;
        rpre[ps][v] = rr;
      }
    }
  }

  // ------------------------------------------------------------------ product
  floatx4 acc[TI][TJ];
#pragma unroll
  for (int ti = 0; ti < TI; ++ti)
#pragma unroll
    for (int tj = 0; tj < TJ; ++tj) acc[ti][tj] = floatx4{0.f, 0.f, 0.f, 0.f};

  float *As = smem;
  float *Bs = smem + BM * (kBK + kKPad);
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int fr = lane & 15, fg = lane >> 4;

  if (GEMM) {
    for (int s = 0; s < p.nseg; ++s) {
      const SegmentP &sg = p.seg[s];
      int64_t kbeg = 0, kend = sg.K;
      if (p.ksplit > 1) {
        const int64_t chunk = ((sg.K + p.ksplit - 1) / p.ksplit + kBK - 1) / kBK * kBK;
        kbeg = ks * chunk;
        kend = kbeg + chunk < sg.K ? kbeg + chunk : sg.K;
      }
      if (kbeg >= kend) continue;
      TileLoader<BM, AK, kBK> la;
      TileLoader<BN, BKM, kBK> lbd;
      la.load(sg.a, b, i0, p.M, kbeg, kend, tid);
      lbd.load(sg.b, b, j0, p.N, kbeg, kend, tid);
      for (int64_t k0 = kbeg; k0 < kend; k0 += kBK) {
        __syncthreads();
        la.store(As, tid);
        lbd.store(Bs, tid);
        __syncthreads();
        if (k0 + kBK < kend) {
          la.load(sg.a, b, i0, p.M, k0 + kBK, kend, tid);
          lbd.load(sg.b, b, j0, p.N, k0 + kBK, kend, tid);
        }
#pragma unroll
        for (int kg = 0; kg < kBK / 16; ++kg) {
          float4 a4[TI], b4[TJ];
#pragma unroll
          for (int ti = 0; ti < TI; ++ti)
            a4[ti] = *reinterpret_cast<const float4 *>(
                As + (wm * WTM + ti * 16 + fr) * (kBK + kKPad) + kg * 16 + 4 * fg);
#pragma unroll
          for (int tj = 0; tj < TJ; ++tj)
            b4[tj] = *reinterpret_cast<const float4 *>(
                Bs + (wn * WTN + tj * 16 + fr) * (kBK + kKPad) + kg * 16 + 4 * fg);
          // independent accumulators back to back, so the matrix pipe overlaps them
#pragma unroll
          for (int ti = 0; ti < TI; ++ti)
#pragma unroll
            for (int tj = 0; tj < TJ; ++tj)
              acc[ti][tj] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[ti].x, b4[tj].x, acc[ti][tj], 0, 0, 0);
#pragma unroll
          for (int ti = 0; ti < TI; ++ti)
#pragma unroll
            for (int tj = 0; tj < TJ; ++tj)
              acc[ti][tj] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[ti].y, b4[tj].y, acc[ti][tj], 0, 0, 0);
#pragma unroll
          for (int ti = 0; ti < TI; ++ti)
#pragma unroll
            for (int tj = 0; tj < TJ; ++tj)
              acc[ti][tj] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[ti].z, b4[tj].z, acc[ti][tj], 0, 0, 0);
#pragma unroll
          for (int ti = 0; ti < TI; ++ti)
#pragma unroll
            for (int tj = 0; tj < TJ; ++tj)
              acc[ti][tj] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[ti].w, b4[tj].w, acc[ti][tj], 0, 0, 0);
        }
      }
    }
    __syncthreads();
    // accumulator tile -> LDS [BM][BN + 4]; lane holds rows 4*fg + v, column fr
    float *Cs = smem;
#pragma unroll
    for (int ti = 0; ti < TI; ++ti)
#pragma unroll
      for (int tj = 0; tj < TJ; ++tj)
#pragma unroll
        for (int v = 0; v < 4; ++v)
          Cs[(wm * WTM + ti * 16 + 4 * fg + v) * (BN + 4) + wn * WTN + tj * 16 + fr] = acc[ti][tj][v];
  }
  __syncthreads();

  // ---------------------------------------------------------------- epilogue
  // Each lane takes four 4-wide column chunks of one row; the chunks of the
  // lanes of one row are interleaved so that a wave's access is contiguous.
  const float *Cs = smem;
  uint32_t run_max = 0u;
  int run_lb = -1;
  int64_t run_gb = -1;
  uint32_t hit_up = 0u, hit_lo = 0u;   // QUANT boundary hits of this thread

#pragma unroll
  for (int ps = 0; ps < NPASS; ++ps) {
    const int row_l = ps * RPP + tid / TPR;
    const int64_t gi = i0 + row_l;
    if (row_l >= BM || gi >= p.M) break;
    const int q = tid % TPR;
    const int64_t lbi = (EPI != EPI_STORE) ? (gi / p.br - lb.bi0) : 0;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int col_l = 4 * q + (BN / 4) * v;
      const int64_t gj = j0 + col_l;
      if (gj >= p.N) continue;
      const bool full = p.vec_out && gj + 3 < p.N;
      float acc4[4] = {0.f, 0.f, 0.f, 0.f};
      if (GEMM) {
        const float4 c = *reinterpret_cast<const float4 *>(Cs + row_l * (BN + 4) + col_l);
        acc4[0] = c.x; acc4[1] = c.y; acc4[2] = c.z; acc4[3] = c.w;
      }
      if (EPI == EPI_STORE) {
        float *cp = p.C + (int64_t)zb * p.cbs + gi * p.ldc + gj;
        const float *dp = p.D ? p.D + (int64_t)b * p.dbs + gi * p.ldd + gj : nullptr;
        const float *cs = p.colscale_tab ? p.colscale_tab[b] : p.colscale;
        float o[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (gj + e < p.N) {
            float val = p.alpha * acc4[e];
            if (dp) val += p.beta * dp[e];
            if (cs) val *= cs[gj + e];
            o[e] = val;
          }
        }
        if (full && (p.ldc % 4 == 0)) {
          *reinterpret_cast<float4 *>(cp) = make_float4(o[0], o[1], o[2], o[3]);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (gj + e < p.N) cp[e] = o[e];
        }
        continue;
      }
      // codec: W~ = D + acc (+ R), D and all codec tensors dense [batch, M, N]
      const int64_t off = (int64_t)b * MN + gi * p.N + gj;
      float w[4];
      // (without a product W~ = W exactly: adding a zero would turn -0 into +0)
      {
        const float4 d = dpre[ps][v];
        if (GEMM) {
          w[0] = d.x + acc4[0]; w[1] = d.y + acc4[1]; w[2] = d.z + acc4[2]; w[3] = d.w + acc4[3];
        } else {
          w[0] = d.x; w[1] = d.y; w[2] = d.z; w[3] = d.w;
        }
        if (p.ef) {
          const float4 rr = rpre[ps][v];
          w[0] += rr.x; w[1] += rr.y; w[2] += rr.z; w[3] += rr.w;
        }
      }
      if (EPI == EPI_AMAX) {
        if (p.transformed) {
          if (full) {
            *reinterpret_cast<float4 *>(p.transformed + off) = make_float4(w[0], w[1], w[2], w[3]);
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (gj + e < p.N) p.transformed[off + e] = w[e];
          }
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (gj + e >= p.N) break;
          const int64_t lbj = (gj + e) / p.bc - lb.bj0;
          const int l = (int)(lbi * lb.nlbj + lbj);
          const uint32_t a = __float_as_uint(w[e]) & 0x7fffffffu;
          if (l != run_lb) {
            if (run_lb >= 0) {
              if (lb.nlb <= kMaxLocalBlocks) atomicMax(&lds_amax[run_lb], run_max);
              else atomicMax(&p.amax[run_gb * kAmaxSlots + slot], run_max);
            }
            run_lb = l;
            run_max = 0u;
            run_gb = (int64_t)b * p.nbr * p.nbc + (gi / p.br) * p.nbc + (gj + e) / p.bc;
          }
          run_max = a > run_max ? a : run_max;
        }
      } else {  // EPI_QUANT
        uint32_t packed = 0u;
        float resid[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (gj + e >= p.N) break;
          float inv, sc;
          const int64_t lbj = (gj + e) / p.bc - lb.bj0;
          const int l = (int)(lbi * lb.nlbj + lbj);
          if (lb.nlb <= kMaxLocalBlocks) {
            inv = lds_inv[l];
            sc = lds_scale[l];
          } else {
            const int64_t gb = (gi / p.br) * p.nbc + (gj + e) / p.bc;
            const float a = __uint_as_float(p.amax[b * (int64_t)p.nbr * p.nbc + gb]);
            inv = e4m3_multiplier(a);
            sc = e4m3_scale(a);
          }
          const float y = w[e] * inv;
          const uint32_t code = e4m3_encode(y);
          packed |= code << (8 * e);
          if (p.hits) {
            hit_up += (code & 0x7fu) == 0x7eu;
            hit_lo += ((code & 0x7fu) == 0u) & (w[e] != 0.0f);
          }
          if (p.ef) resid[e] = w[e] - e4m3_decode(code) * sc;
        }
        uint8_t *cp = p.codes + off;
        if (full && ((off & 3) == 0)) {
          *reinterpret_cast<uint32_t *>(cp) = packed;
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (gj + e < p.N) cp[e] = (uint8_t)(packed >> (8 * e));
        }
        if (p.ef) {
          if (full) {
            *reinterpret_cast<float4 *>(p.ef + off) = make_float4(resid[0], resid[1], resid[2], resid[3]);
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (gj + e < p.N) p.ef[off + e] = resid[e];
          }
        }
      }
    }
  }

  if (EPI == EPI_QUANT && p.hits) e4m3_flush_hits(p.hits + 2 * (int64_t)b, hit_up, hit_lo);
  if (EPI == EPI_AMAX) {
    if (run_lb >= 0) {
      if (lb.nlb <= kMaxLocalBlocks) atomicMax(&lds_amax[run_lb], run_max);
      else atomicMax(&p.amax[run_gb * kAmaxSlots + slot], run_max);
    }
    __syncthreads();
    if (lb.nlb <= kMaxLocalBlocks) {
      for (int l = tid; l < lb.nlb; l += kThreads) {
        const uint32_t v = lds_amax[l];
        if (v != 0u) {
          const int64_t bi = lb.bi0 + l / lb.nlbj, bj = lb.bj0 + l % lb.nlbj;
          atomicMax(&p.amax[((int64_t)b * p.nbr * p.nbc + bi * p.nbc + bj) * kAmaxSlots + slot], v);
        }
      }
    }
  }
}

// One thread per (rank, block), or per block for a shared scale: max over the
// sub-slots (and the ranks), the finished amax and scale s = fl32(amax / 448)
// of every rank, and the sub-slots cleared for the next encode (each slot is
// read by exactly one thread), and the previous encode's slot set cleared.
__global__ void finalize_amax_kernel(uint32_t *raw, int N, int64_t nblk, int shared,
                                     uint32_t *fin, float *scales, uint32_t *clear,
                                     int64_t clear_words) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = t; i < clear_words; i += stride) clear[i] = 0u;
  for (int64_t u = t; u < (shared ? nblk : (int64_t)N * nblk); u += stride) {
    const int b = shared ? 0 : (int)(u / nblk);
    const int64_t blk = shared ? u : u % nblk;
    uint32_t m = 0u;
    for (int r = b; r < (shared ? N : b + 1); ++r) {
      uint32_t *q = raw + ((int64_t)r * nblk + blk) * kAmaxSlots;
      for (int s = 0; s < kAmaxSlots; ++s) {
        m = q[s] > m ? q[s] : m;
        q[s] = 0u;
      }
    }
    const float sc = e4m3_scale(__uint_as_float(m));
    for (int r = b; r < (shared ? N : b + 1); ++r) {
      fin[(int64_t)r * nblk + blk] = m;
      scales[(int64_t)r * nblk + blk] = sc;
    }
  }
}

__global__ void zero_u32_kernel(uint32_t *p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

__global__ void copy_f32_kernel(float *dst, const float *src, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}

KArgs make_args(const TileJob &j) {
  KArgs a{};
  // (a table's pointers are 16-byte aligned: the grouped decode checks them)
  auto op = [](const Operand &o) {
    OperandP r{};
    r.ptr = o.ptr;
    r.ld = o.ld;
    r.bs = o.bs;
    r.vec = (o.ld % 4 == 0) && (o.bs % 4 == 0) && ((reinterpret_cast<uintptr_t>(o.ptr) & 15) == 0);
    r.tab = o.tab;
    return r;
  };
  for (int s = 0; s < 2; ++s) {
    a.seg[s].a = op(j.seg[s].a);
    a.seg[s].b = op(j.seg[s].b);
    a.seg[s].K = j.seg[s].K;
  }
  a.nseg = j.nseg;
  a.ksplit = 1;
  a.M = j.M;
  a.N = j.N;
  a.batch = j.batch;
  a.C = j.C;
  a.ldc = j.ldc;
  a.cbs = j.cbs;
  a.D = j.D;
  a.ldd = j.ldd;
  a.dbs = j.dbs;
  a.alpha = j.alpha;
  a.beta = j.beta;
  a.colscale = j.colscale;
  a.colscale_tab = j.colscale_tab;
  a.amax = j.amax;
  a.codes = j.codes;
  a.hits = j.codes ? j.hits : nullptr;
  a.scales = j.scales;
  a.transformed = j.transformed;
  a.ef = j.ef;
  a.br = j.geom.br;
  a.bc = j.geom.bc;
  a.nbr = j.geom.nbr;
  a.nbc = j.geom.nbc;
  a.shared = j.shared ? 1 : 0;
  auto al16 = [](const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; };
  bool vec = true;
  if (j.C) vec = vec && al16(j.C) && j.ldc % 4 == 0 && j.cbs % 4 == 0;
  if (j.D) vec = vec && al16(j.D) && j.ldd % 4 == 0 && j.dbs % 4 == 0;
  if (j.transformed) vec = vec && al16(j.transformed);
  if (j.ef) vec = vec && al16(j.ef);
  if (j.amax) vec = vec && (j.N % 4 == 0);
  a.vec_out = vec ? 1 : 0;
  return a;
}

template <int BM, int BN, int WM, int WN, bool AK, bool BKM, bool GEMM, int EPI, int BK = 32>
void launch(const KArgs &a, int zdim, hipStream_t st) {
  dim3 grid((unsigned)((a.N + BN - 1) / BN), (unsigned)((a.M + BM - 1) / BM), (unsigned)zdim);
  hipLaunchKernelGGL((tile_kernel<BM, BN, WM, WN, AK, BKM, GEMM, EPI, BK>), grid, dim3(kThreads), 0,
                     st, a);
}

template <int BM, int BN, int WM, int WN, int EPI>
void launch_layouts(const KArgs &a, bool ak, bool bk, int zdim, hipStream_t st) {
  if (ak && bk) launch<BM, BN, WM, WN, true, true, true, EPI>(a, zdim, st);
  else if (ak && !bk) launch<BM, BN, WM, WN, true, false, true, EPI>(a, zdim, st);
  else if (!ak && bk) launch<BM, BN, WM, WN, false, true, true, EPI>(a, zdim, st);
  else launch<BM, BN, WM, WN, false, false, true, EPI>(a, zdim, st);
}

}  // namespace

gift_status launch_tile(gift_ctx *ctx, const TileJob &job) {
  if (job.M <= 0 || job.N <= 0 || job.batch <= 0) return GIFT_OK;
  // per-entry pointer tables (grouped decode): the register-direct update
  // kernel (operands, addend, output) or this file's store tile (operands,
  // column scales), nothing else
  const bool tabs = job_has_tabs(job);
  // the encode's products on the bf16 matrix cores (split operands)
  if (!tabs && job.split3 && job.nseg > 0 && job.amax != nullptr && lr_update_eligible(job))
    return launch_lr_update(ctx, job);
  if (!tabs && job.split3 && job.nseg > 0 && job.amax == nullptr && lr_proj_eligible(job))
    return launch_lr_proj(ctx, job);
  // register-direct kernels for the rank-r update and the projections
  if (job.nseg > 0 && (job.amax != nullptr || job.D != nullptr || job.d_tab != nullptr) &&
      update_kernel_eligible(job))
    return launch_update(ctx, job);
  for (int s = 0; s < job.nseg; ++s)
    if (job.seg[s].a.parts != 1 || job.seg[s].b.parts != 1)
      return set_error(GIFT_EUNSUPPORTED, "split-K partial operand outside the update kernel");
  if (!tabs && job.amax == nullptr && job.nseg > 0 && proj_kernel_eligible(job)) return launch_proj(ctx, job);
  if (tabs && (job.amax != nullptr || job.d_tab != nullptr || job.c_tab != nullptr || job.nseg == 0))
    return set_error(GIFT_EUNSUPPORTED, "internal: pointer tables outside the update and store tile kernels");
  const bool gemm = job.nseg > 0;
  if (job.amax != nullptr && !gemm &&
      stream_eligible(job.M, job.N, job.geom, job.D, job.codes, job.ef, job.transformed))
    return launch_stream_codec(ctx, job);
  KArgs a = make_args(job);
  hipStream_t st = ctx->stream;
  ProfileScope prof(ctx, job.kernel_family);
  if (job.amax == nullptr) {  // EPI_STORE; split K writes partials [batch][ksplit][M][N]
    if (!gemm) return set_error(GIFT_EINVAL, "internal: store tile without a product");
    const bool ak = job.seg[0].a.kmajor, bk = job.seg[0].b.kmajor;
    a.ksplit = job.ksplit > 1 ? job.ksplit : 1;
    const int z = job.batch * a.ksplit;
    if (job.N <= 16) launch_layouts<64, 16, 4, 1, EPI_STORE>(a, ak, bk, z, st);
    else if (job.N <= 32) launch_layouts<64, 32, 4, 1, EPI_STORE>(a, ak, bk, z, st);
    else launch_layouts<64, 64, 2, 2, EPI_STORE>(a, ak, bk, z, st);
    return check_launch("tile_kernel(store)");
  }
  const int epi = job.codes ? EPI_QUANT : EPI_AMAX;
  if (gemm) {
    if (!job.seg[0].a.kmajor || !job.seg[0].b.kmajor ||
        (job.nseg > 1 && (!job.seg[1].a.kmajor || !job.seg[1].b.kmajor)))
      return set_error(GIFT_EINVAL, "internal: codec tile needs K-major operands");
    if (epi == EPI_AMAX) launch<64, 64, 2, 2, true, true, true, EPI_AMAX>(a, job.batch, st);
    else launch<64, 64, 2, 2, true, true, true, EPI_QUANT>(a, job.batch, st);
  } else {
    if (epi == EPI_AMAX) launch<16, 256, 1, 4, true, true, false, EPI_AMAX>(a, job.batch, st);
    else launch<16, 256, 1, 4, true, true, false, EPI_QUANT>(a, job.batch, st);
  }
  return check_launch("tile_kernel(codec)");
}

gift_status launch_zero_u32(gift_ctx *ctx, uint32_t *ptr, int64_t count) {
  if (count <= 0) return GIFT_OK;
  ProfileScope prof(ctx, GIFT_KERNEL_SMALL);
  int64_t blocks = (count + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(zero_u32_kernel, dim3((unsigned)blocks), dim3(256), 0, ctx->stream, ptr, count);
  return check_launch("zero_u32_kernel");
}

gift_status launch_finalize_amax(gift_ctx *ctx, uint32_t *raw, int32_t N, int64_t nblk,
                                 bool shared, uint32_t *fin, float *scales, uint32_t *clear,
                                 int64_t clear_words) {
  const int64_t total = shared ? nblk : (int64_t)N * nblk;
  const int64_t work = total > clear_words ? total : clear_words;
  if (work <= 0) return GIFT_OK;
  int64_t blocks = (work + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  ProfileScope prof(ctx, GIFT_KERNEL_SMALL);
  hipLaunchKernelGGL(finalize_amax_kernel, dim3((unsigned)blocks), dim3(256), 0, ctx->stream,
                     raw, N, nblk, shared ? 1 : 0, fin, scales, clear, clear_words);
  return check_launch("finalize_amax_kernel");
}

gift_status launch_copy_f32(gift_ctx *ctx, float *dst, const float *src, int64_t count) {
  if (count <= 0) return GIFT_OK;
  ProfileScope prof(ctx, GIFT_KERNEL_SMALL);
  int64_t blocks = (count + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(copy_f32_kernel, dim3((unsigned)blocks), dim3(256), 0, ctx->stream, dst, src,
                     count);
  return check_launch("copy_f32_kernel");
}

}  // namespace gift
