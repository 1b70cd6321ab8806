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
// Only tiles on or below the diagonal are computed (A is symmetric); each
// tile is written to both of its mirror positions through an LDS transpose.
// Products of two bfloat16 values are exact in float32 and the sums are
// accumulated in float32 by v_mfma_f32_16x16x32_bf16.  Members of a batch
// (one per factor side with the same dimension) run in one launch.

#include "gift_internal.h"

namespace gift {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kTile = 128;       // output tile (features x features)
constexpr int kKStep = 64;       // tokens per LDS round
constexpr int kRowWords = 32;    // 64 tokens = 32 token-pair words per feature row
constexpr int kThreads = 256;

// LDS layout of one operand: [feature row][32 words], word w of row R holds
// tokens (2w, 2w+1) of that feature.  Words are grouped in 2-word slots
// (4 tokens); slot s of row R is stored at slot s ^ swz(R).  swz(R) is even,
// so the two slots of an aligned 16-byte fragment stay adjacent and in order,
// while the 16 rows written by one store instruction (rows 8 apart) and the 8
// rows read by one 128-byte phase of a fragment load land in different banks.
__device__ __forceinline__ int swz(int row) { return 2 * ((row & 7) ^ ((row >> 3) & 7)); }

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
};

__global__ __launch_bounds__(kThreads) void syrk_bf16_kernel(const SyrkArgs p) {
  constexpr int kOperand = kTile * kRowWords;             // words per operand buffer
  constexpr int kStage = 2 * 2 * kOperand;                // double-buffered A and B
  constexpr int kEpi = kTile * (kTile + 4);
  __shared__ __attribute__((aligned(16))) uint32_t smem[kStage > kEpi ? kStage : kEpi];
  const int tid = threadIdx.x;
  const int member = blockIdx.z;
  // lower-triangle tile (ti >= tj) from the linear block index
  const int x = blockIdx.x;
  int ti = (int)((sqrtf(8.0f * x + 1.0f) - 1.0f) * 0.5f);
  while ((ti + 1) * (ti + 2) / 2 <= x) ++ti;
  while (ti * (ti + 1) / 2 > x) --ti;
  const int tj = x - ti * (ti + 1) / 2;
  const int64_t i0 = (int64_t)ti * kTile, j0 = (int64_t)tj * kTile;
  const uint16_t *X = p.X[member];
  const int64_t T = p.T, dim = p.dim;

  // load mapping: lane -> feature group fgp (8 features, 16 bytes per token
  // row; consecutive lanes read consecutive 16 bytes of a token row) and
  // token quad tq (4 tokens = 2 pair words = one slot).
  const int fgp = tid & 15, tq = tid >> 4;
  uint4 ra[4], rb[4];
  auto load = [&](int64_t t0) {
    const int64_t fi = i0 + 8 * fgp, fj = j0 + 8 * fgp;
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      const int64_t t = t0 + 4 * tq + d;
      const bool tok = t < T;
      ra[d] = (tok && fi < dim) ? *reinterpret_cast<const uint4 *>(X + t * dim + fi) : make_uint4(0, 0, 0, 0);
      rb[d] = (tok && fj < dim) ? *reinterpret_cast<const uint4 *>(X + t * dim + fj) : make_uint4(0, 0, 0, 0);
    }
  };
  auto store = [&](int buf) {
    uint32_t *As = smem + buf * 2 * kOperand;
    uint32_t *Bs = As + kOperand;
    uint32_t w01[8], w23[8];
    pack_pairs(ra[0], ra[1], w01);
    pack_pairs(ra[2], ra[3], w23);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int row = 8 * fgp + e;
      *reinterpret_cast<uint2 *>(As + row * kRowWords + 2 * (tq ^ swz(row))) = make_uint2(w01[e], w23[e]);
    }
    pack_pairs(rb[0], rb[1], w01);
    pack_pairs(rb[2], rb[3], w23);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int row = 8 * fgp + e;
      *reinterpret_cast<uint2 *>(Bs + row * kRowWords + 2 * (tq ^ swz(row))) = make_uint2(w01[e], w23[e]);
    }
  };

  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int fr = lane & 15, fg = lane >> 4;
  floatx4 acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int64_t nsteps = (T + kKStep - 1) / kKStep;
  load(0);
  store(0);
  __syncthreads();
  for (int64_t s = 0; s < nsteps; ++s) {
    const int buf = (int)(s & 1);
    if (s + 1 < nsteps) load((s + 1) * kKStep);
    const uint32_t *As = smem + buf * 2 * kOperand;
    const uint32_t *Bs = As + kOperand;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      // tokens 32 kk + 8 fg .. +7 = slots 8 kk + 2 fg and the next one
      const int slot = 8 * kk + 2 * fg;
      bf16x8 af[4], bfr[4];
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const int row = wm * 64 + a * 16 + fr;
        const uint4 v = *reinterpret_cast<const uint4 *>(As + row * kRowWords + 2 * (slot ^ swz(row)));
        af[a] = __builtin_bit_cast(bf16x8, v);
      }
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int row = wn * 64 + b * 16 + fr;
        const uint4 v = *reinterpret_cast<const uint4 *>(Bs + row * kRowWords + 2 * (slot ^ swz(row)));
        bfr[b] = __builtin_bit_cast(bf16x8, v);
      }
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[a], bfr[b], acc[a][b], 0, 0, 0);
    }
    if (s + 1 < nsteps) store(buf ^ 1);
    __syncthreads();
  }

  // epilogue: tile -> LDS [128][132] -> both mirror positions, coalesced
  float *Cs = reinterpret_cast<float *>(smem);
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        Cs[(wm * 64 + a * 16 + 4 * fg + v) * (kTile + 4) + wn * 64 + b * 16 + fr] = acc[a][b][v] * p.scale;
  __syncthreads();
  float *A = p.A + (int64_t)member * dim * dim;
  for (int q = tid; q < kTile * kTile; q += kThreads) {
    const int r = q / kTile, c = q % kTile;
    const int64_t gi = i0 + r, gj = j0 + c;
    if (gi < dim && gj < dim) A[gi * dim + gj] = Cs[r * (kTile + 4) + c];
  }
  if (ti != tj) {
    for (int q = tid; q < kTile * kTile; q += kThreads) {
      const int r = q / kTile, c = q % kTile;  // output (j0 + r, i0 + c) = tile (c, r)
      const int64_t gi = j0 + r, gj = i0 + c;
      if (gi < dim && gj < dim) A[gi * dim + gj] = Cs[c * (kTile + 4) + r];
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
  ProfileScope prof(ctx, GIFT_KERNEL_SYRK);
  hipLaunchKernelGGL(syrk_bf16_kernel, dim3((unsigned)(nt * (nt + 1) / 2), 1, (unsigned)members),
                     dim3(kThreads), 0, ctx->stream, a);
  return check_launch("syrk_bf16_kernel");
}

}  // namespace gift
