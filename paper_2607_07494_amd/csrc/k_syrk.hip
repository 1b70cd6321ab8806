// Factor statistics A = X^T X / T from bfloat16 tokens on the BF16 matrix
// cores (eq. kfac_fisher_block, eq. impl_A_psd: uncentred second moment).
//
// X is [T, dim] row-major bfloat16 (one token per row).  A workgroup computes
// one 256 x 256 output tile (feature strips i0.. and j0..) with eight waves of
// 128 x 64 each (128 accumulator registers per lane, two waves per SIMD) on
// v_mfma_f32_16x16x32_bf16.  Only tiles on or below the diagonal are
// computed (A is symmetric); each is written to both mirror positions
// straight from the accumulators.
//
// Data path, per stage of 32 tokens:
// * HBM -> LDS by buffer_load_dwordx4 ... lds (no registers, no repacking):
//   each wave instruction fills 1 KiB of LDS (64 lanes x 16 bytes, in lane
//   order) from the lanes' own global addresses.  A stage holds the two
//   strips token-major, [32 tokens][256 features], 16 KiB each; the lanes
//   pick their source so that the 32-byte feature pairs of token row t land
//   at pair slot p ^ sw(t) (see below).  Loads past the last token fall
//   outside the stage's buffer range and arrive as zeros.
// * LDS -> registers by ds_read_b64_tr_b16: a 16-lane group addresses four
//   token rows x 16 features and each lane receives four consecutive tokens
//   of one feature, i.e. half of an MFMA operand fragment (eight tokens of
//   one feature); two reads make a fragment.  The swizzle sw(t) sends the
//   sixteen token rows one read instruction touches to sixteen different
//   pair slots, which spread over all banks.
// * A ring of four stages (four separate LDS arrays per strip, so that the
//   compiler can tell which stage a read depends on) keeps three stages of
//   loads in flight behind the one being multiplied, and the fragments of
//   the next stage are read between the MFMAs of the current one (two
//   fragment register sets).  One barrier per stage orders both the loads
//   (every wave's part of a stage has landed) and the reuse of a slot
//   (every wave has read the stage it held).
// * Diagonal tiles (i0 == j0) load one strip and read both operands from it.
//
// Scheduling: workgroups are handed to the 8 XCDs round-robin by linear id,
// so the launch renumbers them so that each XCD walks a contiguous run of
// (member, tile) pairs, a member's tiles in row-major triangle order; the
// tiles resident on one XCD share a handful of feature strips, fetched into
// that XCD's L2 once.
//
// Products of two bfloat16 values are exact in float32 and the sums are
// accumulated in float32 by the MFMAs, in the same order for every launch
// (deterministic).  Members of a batch (one per factor side with the same
// dimension) run in one launch.

#include "gift_internal.h"

namespace gift {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short shortx4 __attribute__((ext_vector_type(4)));
#define GIFT_LDS __attribute__((address_space(3)))

constexpr int kTile = 256;                    // output tile (features x features)
constexpr int kStageTok = 32;                 // tokens per stage (one MFMA K step)
constexpr int kStripElems = kStageTok * kTile;   // bf16 per strip and stage (16 KiB)
constexpr int kThreads = 512;
constexpr int kXcds = 8;                      // MI355X: 8 XCDs of 32 CUs, each with its own L2

struct SyrkArgs {
  const uint16_t *const *X;  // [members] -> [T, dim] bf16
  float *A;                  // [members, dim, dim]
  int64_t T, dim;
  float scale;               // 1 / T
  int tiles;                 // lower-triangle tiles per member
  int total;                 // members * tiles
  int per_xcd;               // ceil(total / kXcds)
};

// Pair-slot swizzle of token row t (4 bits from token bits 0-1 and 3-4): the
// sixteen rows 8g + 4h + r (g, r = 0..3) of one transposed read get sixteen
// different values.
__device__ __forceinline__ int pair_swizzle(int t) { return (t & 3) | (((t >> 3) & 3) << 2); }

// Wait until at most n of this wave's loads are outstanding (loads complete
// in order), and for this wave's LDS reads; then the workgroup barrier.
__device__ __forceinline__ void wait_loads_barrier(int n) {
  if (n >= 12) asm volatile("s_waitcnt vmcnt(12) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  else if (n >= 8) asm volatile("s_waitcnt vmcnt(8) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  else if (n >= 6) asm volatile("s_waitcnt vmcnt(6) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  else if (n >= 4) asm volatile("s_waitcnt vmcnt(4) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  else if (n >= 2) asm volatile("s_waitcnt vmcnt(2) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  else asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

struct Frags {
  bf16x8 a[8], b[4];
};

template <bool DIAGONAL>
__device__ __forceinline__ void syrk_tile(const SyrkArgs &p, int member, int ti, int tj,
                                          uint16_t *a0, uint16_t *a1, uint16_t *a2, uint16_t *a3,
                                          uint16_t *b0, uint16_t *b1, uint16_t *b2, uint16_t *b3) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int64_t i0 = (int64_t)ti * kTile, j0 = (int64_t)tj * kTile;
  const uint16_t *X = p.X[member];
  const int64_t T = p.T, dim = p.dim;
  const int nst = (int)((T + kStageTok - 1) / kStageTok);
  constexpr int kLoadsPerStage = DIAGONAL ? 2 : 4;   // load instructions per wave and stage

  // Load mapping: wave w fills 1-KiB chunks 2w and 2w + 1 of each strip; a
  // chunk is token rows 2c and 2c + 1.  Lane l writes 16-byte unit pu =
  // l & 31 of row 2c + (l >> 5), which holds the features of logical unit
  // q = 2 ((pu >> 1) ^ sw(t)) + (pu & 1).  Features past dim read whatever
  // lies there (or zeros past the buffer): they only reach outputs that are
  // not stored.
  uint32_t va[2], vb[2];
#pragma unroll
  for (int c2 = 0; c2 < 2; ++c2) {
    const int c = 2 * wave + c2;
    const int t = 2 * c + (lane >> 5);
    const int pu = lane & 31;
    const int q = 2 * ((pu >> 1) ^ pair_swizzle(t)) + (pu & 1);
    va[c2] = (uint32_t)(((int64_t)t * dim + i0 + 8 * q) * 2);
    vb[c2] = (uint32_t)(((int64_t)t * dim + j0 + 8 * q) * 2);
  }
  // a stage at or past the end gets an empty range: its lanes write zeros
  auto load = [&](int s, uint16_t *As, uint16_t *Bs) {
    const int64_t t0 = (int64_t)s * kStageTok;
    const int64_t rest = T - t0 > 0 ? T - t0 : 0;
    const int64_t left = rest < kStageTok ? rest : kStageTok;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(X + t0 * dim), (short)0, (int)(left * dim * 2), 0x00020000);
#pragma unroll
    for (int c2 = 0; c2 < 2; ++c2) {
      const int c = 2 * wave + c2;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (GIFT_LDS void *)(As + c * 512), 16, (int)va[c2], 0, 0, 0);
      if (!DIAGONAL)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (GIFT_LDS void *)(Bs + c * 512), 16, (int)vb[c2], 0, 0, 0);
    }
  };

  // Fragment reads: lane l of group g = l >> 4 (tokens 8g .. 8g + 7 of the
  // stage), j = l & 15 addresses token row 8g + 4h + (j >> 2) and features
  // 4 (j & 3) .. + 3 of a 16-feature pair; it receives tokens 8g + 4h .. +3
  // of feature j.  Fragment a of the A strip (features 128 wm + 16 a ..) is
  // pair 8 wm + a at slot (8 wm + a) ^ swl, swl = sw(row) = (j >> 2) | 4g,
  // i.e. byte rowb + 32 ((8 wm + a) ^ swl).  rowb has bits 5-7 clear, so
  // that is base_a ^ (32 a) with base_a = rowb + 32 ((8 wm) ^ swl): one XOR
  // per fragment (likewise b over the B strip with pair 4 wn + b).
  const int wm = wave >> 2, wn = wave & 3;
  const int g = lane >> 4, j = lane & 15;
  const int swl = (j >> 2) | (g << 2);
  const int rowb = (8 * g + (j >> 2)) * 512 + 8 * (j & 3);
  const int base_a = rowb + 32 * ((8 * wm) ^ swl);
  const int base_b = rowb + 32 * ((4 * wn) ^ swl);

  floatx4 acc[8][4];
#pragma unroll
  for (int a = 0; a < 8; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};

  Frags F0, F1;
  auto frag = [&](const uint16_t *S, int off) {
    const char *c = (const char *)S;
    const shortx4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((GIFT_LDS shortx4 *)(c + off));
    const shortx4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((GIFT_LDS shortx4 *)(c + off + 4 * 512));
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  };
  auto read = [&](Frags &F, const uint16_t *As, const uint16_t *Bs) {
    int ba = base_a, bb = base_b;
    asm volatile("" : "+v"(ba), "+v"(bb));   // keep 2 base registers, not 12 addresses
#pragma unroll
    for (int b = 0; b < 4; ++b) F.b[b] = frag(DIAGONAL ? As : Bs, bb ^ (32 * b));
#pragma unroll
    for (int a = 0; a < 8; ++a) F.a[a] = frag(As, ba ^ (32 * a));
  };
  // the MFMAs of one stage, with the next stage's 24 fragment reads issued
  // one after each of the last 24 MFMAs
  auto mfma_and_read = [&](const Frags &F, Frags &N, const uint16_t *As, const uint16_t *Bs) {
    read(N, As, Bs);
#pragma unroll
    for (int a = 0; a < 8; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b)
        acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(F.a[a], F.b[b], acc[a][b], 0, 0, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
#pragma unroll
    for (int i = 0; i < 24; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  // Stage s lives in slot s % 4.  Step s: barrier on stage s + 1 (its loads
  // have landed everywhere, and every wave has read stage s, so slot s % 4
  // can take stage s + 4), issue the loads of stage s + 4, then the MFMAs of
  // stage s with the reads of stage s + 1 between them.  Loads are issued for
  // every step of the main loop, also past the last stage (empty ranges), so
  // that the number of later loads in flight at each barrier is a constant:
  // three stages after the first one, two in the main loop, and 2, 1, 0 in
  // the (up to three) remaining steps.  The last step also reads a slot
  // (fragments never used) so that every step has one shape.
  load(0, a0, b0);
  load(1, a1, b1);
  load(2, a2, b2);
  load(3, a3, b3);
  wait_loads_barrier(3 * kLoadsPerStage);
  read(F0, a0, b0);
#define GIFT_SYRK_STEP(k, Acur, Bcur, Anx, Bnx, FC, FN, AHEAD, LOAD) \
  {                                                                  \
    wait_loads_barrier((AHEAD) * kLoadsPerStage);                    \
    if (LOAD) load(s + (k) + 4, Acur, Bcur);                         \
    mfma_and_read(FC, FN, Anx, Bnx);                                 \
  }
  int s = 0;
  for (; s + 4 <= nst; s += 4) {
    GIFT_SYRK_STEP(0, a0, b0, a1, b1, F0, F1, 2, true)
    GIFT_SYRK_STEP(1, a1, b1, a2, b2, F1, F0, 2, true)
    GIFT_SYRK_STEP(2, a2, b2, a3, b3, F0, F1, 2, true)
    GIFT_SYRK_STEP(3, a3, b3, a0, b0, F1, F0, 2, true)
  }
  if (s < nst) GIFT_SYRK_STEP(0, a0, b0, a1, b1, F0, F1, 2, false)
  if (s + 1 < nst) GIFT_SYRK_STEP(1, a1, b1, a2, b2, F1, F0, 1, false)
  if (s + 2 < nst) GIFT_SYRK_STEP(2, a2, b2, a3, b3, F0, F1, 0, false)
#undef GIFT_SYRK_STEP
  // no load may still be writing LDS when the workgroup ends
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

  // epilogue straight from the accumulators: lane (fr, fg) of block (a, b)
  // holds rows 4 fg + v, column fr of that 16 x 16 block
  float *A = p.A + (int64_t)member * dim * dim;
  const float sc = p.scale;
  const int fr = lane & 15, fg = lane >> 4;
#pragma unroll
  for (int a = 0; a < 8; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int64_t gi = i0 + wm * 128 + a * 16 + 4 * fg;
      const int64_t gj = j0 + wn * 64 + b * 16 + fr;
      if (gi < dim && gj < dim) {
#pragma unroll
        for (int v = 0; v < 4; ++v) A[(gi + v) * dim + gj] = acc[a][b][v] * sc;
        // mirror: (gj, gi..gi+3) is 16 contiguous bytes (dim % 8 == 0)
        if (!DIAGONAL)
          *reinterpret_cast<float4 *>(A + gj * dim + gi) =
              make_float4(acc[a][b][0] * sc, acc[a][b][1] * sc, acc[a][b][2] * sc, acc[a][b][3] * sc);
      }
    }
}

__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void syrk_bf16_kernel(const SyrkArgs p) {
  // four ring slots per strip, each its own array (128 KiB in total)
  __shared__ __attribute__((aligned(1024))) uint16_t a0[kStripElems], a1[kStripElems], a2[kStripElems],
      a3[kStripElems];
  __shared__ __attribute__((aligned(1024))) uint16_t b0[kStripElems], b1[kStripElems], b2[kStripElems],
      b3[kStripElems];
  // XCD-contiguous renumbering of the linear workgroup id
  const int lin = (int)(blockIdx.x % kXcds) * p.per_xcd + (int)(blockIdx.x / kXcds);
  if (lin >= p.total) return;
  const int member = lin / p.tiles;
  const int x = lin - member * p.tiles;
  // lower-triangle tile (ti >= tj) from the index inside the member
  int ti = (int)((sqrtf(8.0f * x + 1.0f) - 1.0f) * 0.5f);
  while ((ti + 1) * (ti + 2) / 2 <= x) ++ti;
  while (ti * (ti + 1) / 2 > x) --ti;
  const int tj = x - ti * (ti + 1) / 2;
  if (ti == tj)
    syrk_tile<true>(p, member, ti, tj, a0, a1, a2, a3, b0, b1, b2, b3);
  else
    syrk_tile<false>(p, member, ti, tj, a0, a1, a2, a3, b0, b1, b2, b3);
}

}  // namespace

// A[member] = X[member]^T X[member] * scale for all members (device table of
// X pointers).  dim must be a multiple of 8 (16-byte rows).
gift_status launch_syrk_bf16(gift_ctx *ctx, const uint16_t *const *x_table, int members,
                             int64_t T, int64_t dim, float scale, float *A) {
  if (members <= 0) return GIFT_OK;
  if (dim % 8 != 0) return set_error(GIFT_EINVAL, "internal: bf16 statistics need dim % 8 == 0");
  // 32-bit buffer offsets of one stage (32 token rows) and stage counts
  if (dim > (1LL << 24) || T > (1LL << 36))
    return set_error(GIFT_ESHAPE, "internal: statistics shape too large for the bf16 kernel");
  SyrkArgs a{};
  a.X = x_table;
  a.A = A;
  a.T = T;
  a.dim = dim;
  a.scale = scale;
  const int64_t nt = (dim + kTile - 1) / kTile;
  const int64_t total = (int64_t)members * (nt * (nt + 1) / 2);
  if (total > (1LL << 30)) return set_error(GIFT_ESHAPE, "internal: too many statistics tiles");
  a.tiles = (int)(nt * (nt + 1) / 2);
  a.total = (int)total;
  a.per_xcd = (int)((total + kXcds - 1) / kXcds);
  ProfileScope prof(ctx, GIFT_KERNEL_SYRK);
  hipLaunchKernelGGL(syrk_bf16_kernel, dim3((unsigned)(a.per_xcd * kXcds)), dim3(kThreads), 0, ctx->stream, a);
  return check_launch("syrk_bf16_kernel");
}

}  // namespace gift
