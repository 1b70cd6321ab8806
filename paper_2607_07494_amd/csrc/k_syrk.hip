// Factor statistics A = X^T X / T from bfloat16 tokens on the BF16 matrix
// cores (eq. kfac_fisher_block, eq. impl_A_psd: uncentred second moment).
//
// X is [T, dim] row-major bfloat16 (one token per row).  The contraction runs
// over tokens, which are strided in memory, while the MFMA operands need
// consecutive contraction indices per lane.  Each K step of 64 tokens is
// therefore loaded as 16-byte rows of 8 features for four adjacent tokens and
// re-packed in registers into 32-bit (token, token+1) pairs per feature
// before it goes to LDS as [feature][token] with tokens contiguous (8-byte
// stores of two pairs); a lane's MFMA fragment (8 tokens of one feature) is
// then one 16-byte LDS read.
//
// A workgroup computes one 256 x 256 output tile with eight waves of 128 x 64
// each (128 accumulator registers per lane, two waves per SIMD): per 16-byte
// fragment read a wave issues 2.7 MFMAs on average, and the 256-wide strips
// are re-read from L2 half as often as with 128-wide tiles.
// Only tiles on or below the diagonal are computed (A is symmetric); each is
// written to both mirror positions straight from the accumulators.
//
// Scheduling: workgroups are handed to the 8 XCDs round-robin by linear id,
// so the launch renumbers them so that each XCD walks a contiguous run of
// (member, tile) pairs, a member's tiles in row-major triangle order.  The
// ~32 tiles resident on one XCD then share a handful of feature strips that
// advance through the tokens together, and the strips are fetched into that
// XCD's L2 once instead of once per tile.
//
// Products of two bfloat16 values are exact in float32 and the sums are
// accumulated in float32 by v_mfma_f32_16x16x32_bf16.  Members of a batch
// (one per factor side with the same dimension) run in one launch.

#include "gift_internal.h"

namespace gift {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kTile = 256;       // output tile (features x features)
constexpr int kKStep = 64;       // tokens per LDS stage
constexpr int kRowWords = 32;    // 64 tokens = 32 token-pair words per feature row
constexpr int kThreads = 512;
constexpr int kXcds = 8;         // MI355X: 8 XCDs of 32 CUs, each with its own L2

// LDS layout of one operand: [feature row][32 words], word w of row R holds
// tokens (2w, 2w+1) of that feature.  Words are grouped in 2-word slots
// (4 tokens); slot s of row R is stored at slot s ^ swz(R) of physical row
// prow(R).  swz(R) is even, so the two slots of an aligned 16-byte fragment
// stay adjacent and in order.  Bank spread: a fragment read covers 16
// consecutive rows, whose (row parity, swz) pairs are all distinct; a store
// instruction writes rows 8 apart (one feature of each lane's 8), for which
// swz varies with bits 0-2 of the lane's feature group, the 128-byte half of
// the bank window with bit 3 (prow swaps adjacent rows when row bit 6 is
// set), and slot bit 0 with the lane's token quad.
__device__ __forceinline__ int swz(int row) { return 2 * ((row & 7) ^ ((row >> 3) & 7)); }
__device__ __forceinline__ int prow(int row) { return row ^ ((row >> 6) & 1); }

__device__ __forceinline__ void pack_pairs(const uint4 &lo, const uint4 &hi, uint32_t w[8]) {
  // lo: features f..f+7 of token t; hi: the same features of token t+1.
  // w[e] = bf16(t, f+e) | bf16(t+1, f+e) << 16
  const uint32_t l[4] = {lo.x, lo.y, lo.z, lo.w};
  const uint32_t h[4] = {hi.x, hi.y, hi.z, hi.w};
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    w[2 * q] = __builtin_amdgcn_perm(h[q], l[q], 0x05040100u);      // low halves
    w[2 * q + 1] = __builtin_amdgcn_perm(h[q], l[q], 0x07060302u);  // high halves
  }
}

struct SyrkArgs {
  const uint16_t *const *X;  // [members] -> [T, dim] bf16
  float *A;                  // [members, dim, dim]
  int64_t T, dim;
  float scale;               // 1 / T
  int tiles;                 // lower-triangle tiles per member
  int total;                 // members * tiles
  int per_xcd;               // ceil(total / kXcds)
};

__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void syrk_bf16_kernel(const SyrkArgs p) {
  constexpr int kOperand = kTile * kRowWords;   // words per operand and stage (32 KiB)
  constexpr int kStage = 2 * kOperand;          // A and B strips of one stage
  __shared__ __attribute__((aligned(16))) uint32_t smem[2 * kStage];
  const int tid = threadIdx.x;
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
  const int64_t i0 = (int64_t)ti * kTile, j0 = (int64_t)tj * kTile;
  const uint16_t *X = p.X[member];
  const int64_t T = p.T, dim = p.dim;

  // load mapping: thread -> feature group fgp (8 features = 16 bytes of a
  // token row) and token quad tqb (4 tokens = 2 pair words = one slot):
  // tid bits 0-2, 4, 6 -> fgp bits 0-4; tid bits 3, 5, 7, 8 -> tqb bits 0-3.
  // Eight consecutive lanes read 128 contiguous bytes of one token row.
  const int fgp = (tid & 7) | (((tid >> 4) & 1) << 3) | (((tid >> 6) & 1) << 4);
  const int tqb = ((tid >> 3) & 1) | (((tid >> 5) & 1) << 1) | ((tid >> 7) << 2);
  const int64_t fi = i0 + 8 * fgp, fj = j0 + 8 * fgp;
  // Buffer loads: the resource of a stage starts at token t0 and covers only
  // the tokens that exist, so reads past T come back as zero from the range
  // check; a lane whose features lie past dim gets an offset beyond any
  // stage's range and reads zeros too.
  constexpr uint32_t kOutside = 0x40000000u;   // > 64 * dim * 2 for dim < 2^23
  const uint32_t row_bytes = (uint32_t)dim * 2u;
  const uint32_t offi = fi < dim ? (uint32_t)(4 * tqb) * row_bytes + (uint32_t)fi * 2u : kOutside;
  const uint32_t offj = fj < dim ? (uint32_t)(4 * tqb) * row_bytes + (uint32_t)fj * 2u : kOutside;
  uint4 ra[4], rb[4];
  auto load = [&](int64_t t0) {
    const int64_t left = T - t0 < kKStep ? T - t0 : kKStep;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(X + t0 * dim), (short)0, (int)(left * dim * 2), 0x00020000);
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      const uint32_t tok = (uint32_t)d * row_bytes;
      ra[d] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rs, (int)(offi + tok), 0, 0));
      rb[d] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rs, (int)(offj + tok), 0, 0));
    }
  };
  auto store = [&](int buf) {
    uint32_t *As = smem + buf * kStage;
    uint32_t *Bs = As + kOperand;
    const int tq = tqb;
    uint32_t w01[8], w23[8];
    pack_pairs(ra[0], ra[1], w01);
    pack_pairs(ra[2], ra[3], w23);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int row = 8 * fgp + e;
      *reinterpret_cast<uint2 *>(As + prow(row) * kRowWords + 2 * (tq ^ swz(row))) = make_uint2(w01[e], w23[e]);
    }
    pack_pairs(rb[0], rb[1], w01);
    pack_pairs(rb[2], rb[3], w23);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int row = 8 * fgp + e;
      *reinterpret_cast<uint2 *>(Bs + prow(row) * kRowWords + 2 * (tq ^ swz(row))) = make_uint2(w01[e], w23[e]);
    }
  };

  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;
  const int fr = lane & 15, fg = lane >> 4;
  floatx4 acc[8][4];
#pragma unroll
  for (int a = 0; a < 8; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int64_t nsteps = (T + kKStep - 1) / kKStep;
  load(0);
  store(0);
  __syncthreads();
  for (int64_t s = 0; s < nsteps; ++s) {
    const int buf = (int)(s & 1);
    if (s + 1 < nsteps) load((s + 1) * kKStep);
    const uint32_t *As = smem + buf * kStage;
    const uint32_t *Bs = As + kOperand;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      // tokens 32 kk + 8 fg .. +7 = slots 8 kk + 2 fg and the next one
      const int slot = 8 * kk + 2 * fg;
      bf16x8 af[8], bfr[4];
#pragma unroll
      for (int a = 0; a < 8; ++a) {
        const int row = wm * 128 + a * 16 + fr;
        const uint4 v = *reinterpret_cast<const uint4 *>(As + prow(row) * kRowWords + 2 * (slot ^ swz(row)));
        af[a] = __builtin_bit_cast(bf16x8, v);
      }
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int row = wn * 64 + b * 16 + fr;
        const uint4 v = *reinterpret_cast<const uint4 *>(Bs + prow(row) * kRowWords + 2 * (slot ^ swz(row)));
        bfr[b] = __builtin_bit_cast(bf16x8, v);
      }
#pragma unroll
      for (int a = 0; a < 8; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[a], bfr[b], acc[a][b], 0, 0, 0);
    }
    if (s + 1 < nsteps) store(buf ^ 1);
    __syncthreads();
  }

  // epilogue straight from the accumulators: lane (fr, fg) of block (a, b)
  // holds rows 4 fg + v, column fr of that 16 x 16 block
  float *A = p.A + (int64_t)member * dim * dim;
  const float sc = p.scale;
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
        if (ti != tj)
          *reinterpret_cast<float4 *>(A + gj * dim + gi) =
              make_float4(acc[a][b][0] * sc, acc[a][b][1] * sc, acc[a][b][2] * sc, acc[a][b][3] * sc);
      }
    }
}

}  // namespace

// A[member] = X[member]^T X[member] * scale for all members (device table of
// X pointers).  dim must be a multiple of 8 (16-byte rows).
gift_status launch_syrk_bf16(gift_ctx *ctx, const uint16_t *const *x_table, int members,
                             int64_t T, int64_t dim, float scale, float *A) {
  if (members <= 0) return GIFT_OK;
  if (dim % 8 != 0) return set_error(GIFT_EINVAL, "internal: bf16 statistics need dim % 8 == 0");
  SyrkArgs a;
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
