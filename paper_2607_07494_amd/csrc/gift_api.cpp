// C ABI of the GIFT codec: argument validation, object lifetime and the
// kernel sequence of each call.
//
// Transform in rank-r form (Sec. IV-A, V-A, V-B; Algorithm 1).  With
// S_A^-1 = I + U_A C_A U_A^T (n x n) and S_G^-1 = I + U_G C_G U_G^T (m x m),
// the encode of one rank's W computes
//
//   INPUT   W~ = W + P (C_A U_A^T),                 P = W U_A          (m x r)
//   OUTPUT  W~ = W + (U_G C_G) Q,                   Q = U_G^T W        (r x n)
//   BOTH    W~ = W + (U_G C_G) Q + L2 U_A^T,        L2 = (P + U_G C_G K) C_A,
//                                                   K = U_G^T P        (r x r)
//
// i.e. W~ = S_G^-1 W S_A^-1 as one rank-r (rank-2r) update of W.  Each update
// runs twice: once fused with the block amax, once fused with the
// quantization (the scale needs the finished amax of the whole block, so W~
// is recomputed rather than written to memory).  The decode applies the same
// form with the inverse coefficients C' to the rank mean.

#include <math.h>
#include <string.h>

#include <mutex>
#include <new>
#include <string>

#include "gift_internal.h"

// Device scratch of gift_encode_noalloc, the entry point for callers that
// cannot allocate device memory.  Every device the library runs on holds its
// own copy from the moment the code object is loaded there until the process
// ends.  Host code never takes this array's address directly (on the host the
// name is only a stand-in for the symbol): noalloc_scratch() looks the device
// address up once per device with hipGetSymbolAddress and the kernels receive
// that pointer.
static __device__ __align__(256) unsigned char scratch[GIFT_NOALLOC_SCRATCH_BYTES];

namespace gift {

namespace {
thread_local std::string g_last_error;
}

gift_status set_error(gift_status st, const std::string &msg) {
  g_last_error = msg;
  return st;
}

gift_status hip_error(hipError_t e, const char *what) {
  return set_error(GIFT_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

gift_status check_launch(const char *what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_error(e, what);
  return GIFT_OK;
}

gift_status bind_device(gift_ctx *ctx) {
  if (ctx->device >= 0) return GIFT_OK;
  int dev = -1;
  GIFT_HIP_TRY(hipGetDevice(&dev));
  ctx->device = dev;
  return GIFT_OK;
}

gift_status grow_buffer(gift_ctx *ctx, Workspace &w, size_t bytes, void **out) {
  bytes = (bytes + 255) & ~(size_t)255;
  if (bytes == 0) bytes = 256;
  if (bytes > w.bytes) {
    if (w.ptr) {
      GIFT_HIP_TRY(hipStreamSynchronize(ctx->stream));
      GIFT_HIP_TRY(hipFree(w.ptr));
      w.ptr = nullptr;
      w.bytes = 0;
    }
    void *p = nullptr;
    hipError_t e = hipMalloc(&p, bytes);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return set_error(GIFT_ENOMEM, "workspace: hipMalloc of " + std::to_string(bytes) + " bytes failed");
    }
    w.ptr = p;
    w.bytes = bytes;
  }
  *out = w.ptr;
  return GIFT_OK;
}

gift_status workspace(gift_ctx *ctx, size_t bytes, void **out) { return grow_buffer(ctx, ctx->ws, bytes, out); }

gift_status upload_table(gift_ctx *ctx, int kind, const void *owner, const void *host, size_t bytes,
                         void **dev) {
  TableSlot &t = ctx->tables[std::make_pair(kind, owner)];
  if (t.valid && t.last.size() == bytes && memcmp(t.last.data(), host, bytes) == 0) {
    *dev = t.dev.ptr;
    return GIFT_OK;
  }
  t.valid = false;
  void *d = nullptr;
  gift_status st = grow_buffer(ctx, t.dev, bytes, &d);
  if (st != GIFT_OK) return st;
  if (t.copied) {
    // the pinned buffer is rewritten below: its last copy must have run
    hipError_t q = hipEventQuery(t.copied);
    if (q == hipErrorNotReady) {
      GIFT_HIP_TRY(hipEventSynchronize(t.copied));
    } else if (q != hipSuccess) {
      return hip_error(q, "upload_table: hipEventQuery");
    }
  } else {
    GIFT_HIP_TRY(hipEventCreateWithFlags(&t.copied, hipEventDisableTiming));
  }
  if (t.pinned_bytes < bytes) {
    if (t.pinned) GIFT_HIP_TRY(hipHostFree(t.pinned));
    t.pinned = nullptr;
    t.pinned_bytes = 0;
    void *p = nullptr;
    hipError_t e = hipHostMalloc(&p, bytes, 0);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return set_error(GIFT_ENOMEM, "upload_table: hipHostMalloc of " + std::to_string(bytes) + " bytes failed");
    }
    t.pinned = p;
    t.pinned_bytes = bytes;
  }
  memcpy(t.pinned, host, bytes);
  GIFT_HIP_TRY(hipMemcpyAsync(d, t.pinned, bytes, hipMemcpyHostToDevice, ctx->stream));
  GIFT_HIP_TRY(hipEventRecord(t.copied, ctx->stream));
  t.last.assign(static_cast<const char *>(host), static_cast<const char *>(host) + bytes);
  t.valid = true;
  *dev = d;
  return GIFT_OK;
}

gift_status amax_slots(gift_ctx *ctx, size_t words, uint32_t **cur, uint32_t **other,
                       size_t *other_dirty) {
  if (words > ctx->slot_words || ctx->slots_unknown) {
    if (words > ctx->slot_words) {
      size_t cap = ctx->slot_words ? ctx->slot_words : 4096;
      while (cap < words) cap *= 2;
      if (ctx->slots.ptr) {
        GIFT_HIP_TRY(hipStreamSynchronize(ctx->stream));
        GIFT_HIP_TRY(hipFree(ctx->slots.ptr));
        ctx->slots.ptr = nullptr;
        ctx->slots.bytes = 0;
        ctx->slot_words = 0;
      }
      void *p = nullptr;
      if (hipMalloc(&p, 2 * cap * sizeof(uint32_t)) != hipSuccess) {
        (void)hipGetLastError();
        return set_error(GIFT_ENOMEM, "amax slots: hipMalloc failed");
      }
      ctx->slots.ptr = p;
      ctx->slots.bytes = 2 * cap * sizeof(uint32_t);
      ctx->slot_words = cap;
    }
    gift_status st = launch_zero_u32(ctx, static_cast<uint32_t *>(ctx->slots.ptr), (int64_t)(2 * ctx->slot_words));
    if (st != GIFT_OK) return st;
    ctx->slot_dirty[0] = ctx->slot_dirty[1] = 0;
    ctx->slots_unknown = false;
  }
  uint32_t *base = static_cast<uint32_t *>(ctx->slots.ptr);
  const int s = ctx->slot_set;
  *cur = base + (size_t)s * ctx->slot_words;
  *other = base + (size_t)(1 - s) * ctx->slot_words;
  *other_dirty = ctx->slot_dirty[1 - s];
  ctx->slots_unknown = true;   // until amax_slots_done
  return GIFT_OK;
}

void amax_slots_done(gift_ctx *ctx, size_t left) {
  const int s = ctx->slot_set;
  ctx->slot_dirty[s] = left;
  ctx->slot_dirty[1 - s] = 0;
  ctx->slot_set = 1 - s;
  ctx->slots_unknown = false;
}

ProfileScope::ProfileScope(gift_ctx *c, int k) : ctx(c), kernel(k) {
  if (!ctx || !ctx->profile || ctx->no_alloc_call || !((ctx->profile_mask >> kernel) & 1u)) return;
  hipEvent_t start = nullptr;
  auto grab = [&]() -> hipEvent_t {
    if (!ctx->event_pool.empty()) {
      hipEvent_t e = ctx->event_pool.back();
      ctx->event_pool.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  };
  start = grab();
  stop = grab();
  if (!start || !stop) {
    stop = nullptr;
    return;
  }
  (void)hipEventRecord(start, ctx->stream);
  ctx->prof.push_back(ProfileRec{kernel, start, stop});
}

ProfileScope::~ProfileScope() {
  if (stop) (void)hipEventRecord(stop, ctx->stream);
}

BlockGeom block_geom(int64_t m, int64_t n, int32_t block_rows, int32_t block_cols) {
  BlockGeom g;
  g.br = block_rows <= 0 ? m : (block_rows < m ? block_rows : m);
  g.bc = block_cols <= 0 ? n : (block_cols < n ? block_cols : n);
  g.nbr = (int32_t)((m + g.br - 1) / g.br);
  g.nbc = (int32_t)((n + g.bc - 1) / g.bc);
  return g;
}

namespace {

constexpr int64_t kMaxRows = 65535LL * 16;     // grid.y limit of the 16-row tiles
constexpr int64_t kMaxCols = (1LL << 31) - 1;
constexpr int32_t kMaxRanks = 65535;            // grid.z limit
constexpr int64_t kMaxCholBlock = 8192;        // one workgroup factors a block
constexpr int32_t kMaxRank = 512;               // subspace block k = 2r <= 1024

gift_status drain_profile(gift_ctx *ctx) {
  if (ctx->prof.empty()) return GIFT_OK;
  GIFT_HIP_TRY(hipStreamSynchronize(ctx->stream));
  for (const ProfileRec &r : ctx->prof) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.start, r.stop) == hipSuccess) {
      ctx->prof_ms[r.kernel] += ms;
      ctx->prof_launches[r.kernel] += 1;
    }
    ctx->event_pool.push_back(r.start);
    ctx->event_pool.push_back(r.stop);
  }
  ctx->prof.clear();
  return GIFT_OK;
}

bool side_in(int32_t sides, int32_t s) { return (sides & s) != 0; }

size_t a256(size_t b) { return (b + 255) & ~(size_t)255; }

gift_status check_matrix_dims(int64_t m, int64_t n) {
  if (m <= 0 || n <= 0) return set_error(GIFT_ESHAPE, "m and n must be positive");
  if (m > kMaxRows) return set_error(GIFT_ESHAPE, "m exceeds the supported maximum (1048560)");
  if (n > kMaxCols) return set_error(GIFT_ESHAPE, "n exceeds the supported maximum (2^31-1)");
  return GIFT_OK;
}

bool al16p(const void *q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; }

// The encode recomputes W~ in its quantize pass, instead of storing it and
// reading it back, when the split-bf16 update kernel takes the job: with
// cheap products, reading W again (4 B per element) costs less than writing
// and reading W~ (8 B).  Conditions mirror lr_update_eligible.
bool encode_recomputes(const gift_factor *f, int64_t n, const float *grads, const float *ef,
                       const uint8_t *codes, const float *transformed) {
  const bool useA = side_in(f->sides, GIFT_SIDE_INPUT) && f->A.r > 0;
  const bool useG = side_in(f->sides, GIFT_SIDE_OUTPUT) && f->G.r > 0;
  if (!useA && !useG) return false;
  if (useA && useG && f->A.r != f->G.r) return false;
  // the split-bf16 update kernels take one rank's slice within a 32-bit
  // buffer range; larger matrices store W~ and quantize it in a second pass
  if (f->m * n >= (1LL << 29)) return false;
  const int K = useA ? f->A.r : f->G.r;
  if (K > 128 || K % 4 != 0 || n % 4 != 0) return false;
  // both sides at rank 96 or 128 without a residual: the rank-2r update is
  // bound by the matrix cores, so the AMAX pass (sweep variant) stores W~
  // and the quantize pass streams it rather than forming it again
  if (useA && useG && K >= 96 && n % 128 == 0 && !ef) return false;
  return al16p(grads) && (!ef || al16p(ef)) && (!transformed || al16p(transformed)) &&
         (reinterpret_cast<uintptr_t>(codes) & 3) == 0;
}

// W~ = W + (low-rank part of the transform) for all N ranks.  Fills the
// projection buffers in `ws` and returns the update as a tile job (without
// epilogue fields); side inverse=true builds the decode's S_G M S_A update.
struct LowRankPlan {
  TileJob upd;
  bool active = false;
};

// The two-sided form's products with small grids (K = U_G^T P always, and
// W^T U_G over few ranks: 4 to 64 tiles of 64 x 64) split their contraction
// over the rows into partials, summed in order: enough workgroups to fill
// the GPU.
int small_split(int64_t M, int64_t Nc, int64_t batch, int64_t K) {
  const int64_t tiles = (M + 63) / 64 * ((Nc + 63) / 64) * batch;
  int ks = 1;
  while (ks < 16 && tiles * ks < 512 && K / (2 * ks) >= 64) ks *= 2;
  return ks;
}

gift_status plan_low_rank(gift_ctx *ctx, const gift_factor *f, const float *W, int32_t N,
                          int64_t m, int64_t n, bool inverse, char *ws, size_t *used,
                          LowRankPlan *plan) {
  const Side &A = f->A;
  const Side &G = f->G;
  const bool useA = side_in(f->sides, GIFT_SIDE_INPUT) && A.r > 0;
  const bool useG = side_in(f->sides, GIFT_SIDE_OUTPUT) && G.r > 0;
  plan->active = useA || useG;
  if (!plan->active) return GIFT_OK;
  const int64_t mn = m * n;
  // input side alone: the projection may split its contraction into partials
  // that the update kernel sums (same conditions as that kernel's)
  // (the encode's split-bf16 projection has its own partial count)
  const bool aligned = (reinterpret_cast<uintptr_t>(W) & 15) == 0;
  // (both sides: the decode's projection alone, summed before its two uses)
  const bool pp_ok = useA && (!useG || inverse) && aligned && n % 4 == 0 &&
                     (A.r == 16 || A.r == 32 || A.r == 64 || A.r == 128);
  const int pparts = !pp_ok ? 1 : (inverse ? proj_parts(m, n, A.r, N) : lr_proj_parts(m, n, N));
  // (the in-order sum reads 16-byte groups: a partial's size a multiple of 4)
  // The encode's U_G^T W at rank 64 or 128 takes the split-bf16 transposed
  // projection with its own partial count.
  const int pt_parts = useG && !inverse && aligned && al16p(G.Ut) ? lr_projT_parts(n, m, G.r, N) : 0;
  const int qsplit = pt_parts > 0 ? pt_parts : useG && (n * G.r) % 4 == 0 ? small_split(n, G.r, N, m) : 1;
  // the encode's K at ranks 64 / 128 as Kᵀ = Pᵀ U_G on the same transposed
  // split-bf16 projection (Kᵀ [r_A][r_G] then feeds L2 K-major)
  const int kt_parts = useA && useG && !inverse && al16p(G.Ut) ? lr_projT_parts(A.r, m, G.r, N) : 0;
  const int ksplit_k = kt_parts > 0                                  ? kt_parts
                       : useA && useG && ((int64_t)G.r * A.r) % 4 == 0 ? small_split(G.r, A.r, N, m)
                                                                       : 1;
  size_t off = 0;
  float *P = nullptr, *Qm = nullptr, *Km = nullptr, *L2 = nullptr, *Psum = nullptr;
  float *Qpart = nullptr, *Kpart = nullptr;
  if (useA) {
    P = reinterpret_cast<float *>(ws + off);
    off += a256(sizeof(float) * N * pparts * m * A.r);
  }
  // the encode sums the projection's partials once (the update then reads
  // one P per column range instead of all partials), and so does the
  // two-sided decode (K and L2 read P)
  const bool presum = (!inverse || useG) && pparts > 1;
  if (presum) {
    Psum = reinterpret_cast<float *>(ws + off);
    off += a256(sizeof(float) * N * m * A.r);
  }
  if (useG) {
    Qm = reinterpret_cast<float *>(ws + off);
    off += a256(sizeof(float) * N * n * G.r);
  }
  if (useA && useG) {
    Km = reinterpret_cast<float *>(ws + off);
    off += a256(sizeof(float) * N * G.r * A.r);
    L2 = reinterpret_cast<float *>(ws + off);
    off += a256(sizeof(float) * N * m * A.r);
  }
  if (qsplit > 1) {
    Qpart = reinterpret_cast<float *>(ws + off);
    off += a256(sizeof(float) * N * qsplit * n * G.r);
  }
  if (ksplit_k > 1) {
    Kpart = reinterpret_cast<float *>(ws + off);
    off += a256(sizeof(float) * N * ksplit_k * G.r * A.r);
  }
  // the forward update's column operands as the sweep kernel's LDS images:
  // input side alone, C_A U_A^T (shared); both sides at one rank, Q of each
  // rank and U_A^T (shared)
  const bool two_img = !inverse && useA && useG && A.r == G.r && lr_col_image_bytes(n, A.r) > 0;
  const size_t img_bytes = !inverse && useA && (!useG || two_img) ? lr_col_image_bytes(n, A.r) : 0;
  const size_t qimg_bytes = two_img ? lr_col_image_bytes(n, G.r) : 0;
  void *img = nullptr, *qimg = nullptr;
  if (img_bytes) {
    img = ws + off;
    off += a256(img_bytes);
  }
  if (qimg_bytes) {
    qimg = ws + off;
    off += a256(qimg_bytes * N);
  }
  *used = off;
  if (ws == nullptr) return GIFT_OK;  // sizing pass
  gift_status st;
  const float *UcG = inverse ? G.Uci : G.Uc;
  if (useA) {  // P = W U_A
    TileJob j;
    j.nseg = 1;
    j.seg[0].a = Operand{W, n, mn, true};
    j.seg[0].b = Operand{A.Ut, n, 0, true};
    j.seg[0].K = n;
    j.M = m;
    j.N = A.r;
    j.batch = N;
    j.C = P;
    j.ldc = A.r;
    j.cbs = m * A.r;
    j.ksplit = pparts;
    j.split3 = !inverse;
    j.kernel_family = inverse ? GIFT_KERNEL_DECODE_PROJECT : GIFT_KERNEL_PROJECT;
    if ((st = launch_tile(ctx, j)) != GIFT_OK) return st;
    if (presum &&
        (st = launch_lr_psum(ctx, P, Psum, pparts, m * A.r, N,
                            inverse ? GIFT_KERNEL_DECODE_PROJECT : GIFT_KERNEL_PROJECT)) != GIFT_OK)
      return st;
  }
  if (useG) {  // Qm = W^T U_G  (Q^T, n x r)
    TileJob j;
    j.nseg = 1;
    j.seg[0].a = Operand{W, n, mn, false};
    j.seg[0].b = Operand{G.Ut, m, 0, true};
    j.seg[0].K = m;
    j.M = n;
    j.N = G.r;
    j.batch = N;
    j.C = qsplit > 1 ? Qpart : Qm;
    j.ldc = G.r;
    j.cbs = n * G.r;
    j.ksplit = qsplit;
    j.kernel_family = inverse ? GIFT_KERNEL_DECODE_PROJECT : GIFT_KERNEL_PROJECT;
    j.split3 = pt_parts > 0;
    if ((st = j.split3 ? launch_lr_projT(ctx, j) : launch_tile(ctx, j)) != GIFT_OK) return st;
    if (qsplit > 1 && (st = launch_lr_psum(ctx, Qpart, Qm, qsplit, n * G.r, N, j.kernel_family)) != GIFT_OK)
      return st;
  }
  if (useA && useG) {
    {  // K = U_G^T P  (r_G x r_A), or Kᵀ = Pᵀ U_G  (r_A x r_G)
      TileJob j;
      j.nseg = 1;
      if (kt_parts > 0) {
        j.seg[0].a = Operand{presum ? Psum : P, A.r, m * A.r, false};
        j.seg[0].b = Operand{G.Ut, m, 0, true};
        j.M = A.r;
        j.N = G.r;
        j.ldc = G.r;
        j.split3 = true;
      } else {
        j.seg[0].a = Operand{G.Ut, m, 0, true};
        j.seg[0].b = Operand{presum ? Psum : P, A.r, m * A.r, false};
        j.M = G.r;
        j.N = A.r;
        j.ldc = A.r;
      }
      j.seg[0].K = m;
      j.batch = N;
      j.C = ksplit_k > 1 ? Kpart : Km;
      j.cbs = (int64_t)G.r * A.r;
      j.ksplit = ksplit_k;
      j.kernel_family = inverse ? GIFT_KERNEL_DECODE_PROJECT : GIFT_KERNEL_PROJECT;
      if ((st = kt_parts > 0 ? launch_lr_projT(ctx, j) : launch_tile(ctx, j)) != GIFT_OK) return st;
      if (ksplit_k > 1 &&
          (st = launch_lr_psum(ctx, Kpart, Km, ksplit_k, (int64_t)G.r * A.r, N, j.kernel_family)) != GIFT_OK)
        return st;
    }
    {  // L2 = (P + U_G C_G K) C_A
      TileJob j;
      j.nseg = 1;
      j.seg[0].a = Operand{UcG, G.r, 0, true};
      j.seg[0].b = kt_parts > 0 ? Operand{Km, G.r, (int64_t)G.r * A.r, true}
                                : Operand{Km, A.r, (int64_t)G.r * A.r, false};
      j.seg[0].K = G.r;
      j.M = m;
      j.N = A.r;
      j.batch = N;
      j.C = L2;
      j.ldc = A.r;
      j.cbs = m * A.r;
      j.D = presum ? Psum : P;
      j.ldd = A.r;
      j.dbs = m * A.r;
      j.beta = 1.f;
      j.colscale = inverse ? A.c_inv : A.c_fwd;
      j.split3 = kt_parts > 0;   // the split-bf16 projection kernel with its addend and scales
      j.kernel_family = inverse ? GIFT_KERNEL_DECODE_PROJECT : GIFT_KERNEL_PROJECT;
      if ((st = launch_tile(ctx, j)) != GIFT_OK) return st;
    }
  }
  TileJob &u = plan->upd;
  u.M = m;
  u.N = n;
  u.batch = N;
  u.nseg = 0;
  u.split3 = !inverse;
  if (useG) {  // (U_G C_G) Q, with B(k, j) = Q[k][j] = Qm[j][k]
    Segment &s = u.seg[u.nseg++];
    s.a = Operand{UcG, G.r, 0, true};
    s.b = Operand{Qm, G.r, n * G.r, true};
    s.K = G.r;
  }
  if (useA) {
    Segment &s = u.seg[u.nseg++];
    if (useG) {  // L2 U_A^T
      s.a = Operand{L2, A.r, m * A.r, true};
      s.b = Operand{A.U, A.r, 0, true};
      if (two_img) {
        u.col_img = qimg;   // segment 0: Q of each rank
        u.img_bs = (int64_t)qimg_bytes;
        u.col_img2 = img;   // segment 1: U_A^T
        if ((st = launch_lr_col_image(ctx, Qm, G.r, n, (int)G.r, qimg, N, n * G.r)) != GIFT_OK ||
            (st = launch_lr_col_image(ctx, A.U, A.r, n, (int)A.r, img)) != GIFT_OK)
          return st;
      }
    } else if (presum) {  // P (C_A U_A^T), P already summed
      s.a = Operand{Psum, A.r, m * A.r, true, 1};
      s.b = Operand{A.Uc, A.r, 0, true};
      u.col_img = img;
    } else {  // P (C_A U_A^T), P summed from its partials
      s.a = Operand{P, A.r, m * A.r, true, pparts};
      s.b = Operand{inverse ? A.Uci : A.Uc, A.r, 0, true};
      if (!inverse) u.col_img = img;
    }
    s.K = A.r;
    if (!useG && u.col_img && (st = launch_lr_col_image(ctx, A.Uc, A.r, n, (int)A.r, img)) != GIFT_OK) return st;
  }
  return GIFT_OK;
}

}  // namespace
}  // namespace gift

using namespace gift;

extern "C" {

int32_t gift_abi_version(void) { return GIFT_ABI_VERSION; }

const char *gift_last_error(void) { return g_last_error.c_str(); }

gift_status gift_ctx_create(void *hip_stream, gift_ctx **out) {
  if (!out) return set_error(GIFT_EINVAL, "gift_ctx_create: out is NULL");
  gift_ctx *c = new (std::nothrow) gift_ctx();
  if (!c) return set_error(GIFT_ENOMEM, "gift_ctx_create: out of host memory");
  c->stream = static_cast<hipStream_t>(hip_stream);
  *out = c;
  return GIFT_OK;
}

gift_status gift_ctx_set_stream(gift_ctx *ctx, void *hip_stream) {
  if (!ctx) return set_error(GIFT_EINVAL, "gift_ctx_set_stream: ctx is NULL");
  // the workspace and the amax sub-slots are ordered by the old stream
  if (ctx->device >= 0 && ctx->stream != static_cast<hipStream_t>(hip_stream))
    GIFT_HIP_TRY(hipStreamSynchronize(ctx->stream));
  ctx->stream = static_cast<hipStream_t>(hip_stream);
  return GIFT_OK;
}

void gift_ctx_destroy(gift_ctx *ctx) {
  if (!ctx) return;
  if (ctx->device >= 0) {
    (void)hipStreamSynchronize(ctx->stream);
    for (const ProfileRec &r : ctx->prof) {
      (void)hipEventDestroy(r.start);
      (void)hipEventDestroy(r.stop);
    }
    for (hipEvent_t e : ctx->event_pool) (void)hipEventDestroy(e);
    if (ctx->ws.ptr) (void)hipFree(ctx->ws.ptr);
    if (ctx->slots.ptr) (void)hipFree(ctx->slots.ptr);
    if (ctx->xform.ptr) (void)hipFree(ctx->xform.ptr);
    for (auto &kv : ctx->tables) {
      if (kv.second.dev.ptr) (void)hipFree(kv.second.dev.ptr);
      if (kv.second.pinned) (void)hipHostFree(kv.second.pinned);
      if (kv.second.copied) (void)hipEventDestroy(kv.second.copied);
    }
  }
  delete ctx;
}

gift_status gift_ctx_set_statistics_event(gift_ctx *ctx, void *hip_event) {
  if (!ctx) return set_error(GIFT_EINVAL, "gift_ctx_set_statistics_event: ctx is NULL");
  ctx->stats_event = static_cast<hipEvent_t>(hip_event);
  return GIFT_OK;
}

gift_status gift_ctx_profile_enable(gift_ctx *ctx, int32_t enable) {
  if (!ctx) return set_error(GIFT_EINVAL, "gift_ctx_profile_enable: ctx is NULL");
  ctx->profile = enable != 0;
  return GIFT_OK;
}

gift_status gift_ctx_profile_select(gift_ctx *ctx, uint32_t family_mask) {
  if (!ctx) return set_error(GIFT_EINVAL, "gift_ctx_profile_select: ctx is NULL");
  ctx->profile_mask = family_mask;
  return GIFT_OK;
}

gift_status gift_ctx_profile_read(gift_ctx *ctx, int32_t kernel, int64_t *launches,
                                  double *total_ms) {
  if (!ctx || !launches || !total_ms)
    return set_error(GIFT_EINVAL, "gift_ctx_profile_read: NULL argument");
  if (kernel < 0 || kernel >= GIFT_KERNEL_COUNT)
    return set_error(GIFT_EINVAL, "gift_ctx_profile_read: unknown kernel family");
  gift_status st = drain_profile(ctx);
  if (st != GIFT_OK) return st;
  *launches = ctx->prof_launches[kernel];
  *total_ms = ctx->prof_ms[kernel];
  return GIFT_OK;
}

gift_status gift_ctx_profile_reset(gift_ctx *ctx) {
  if (!ctx) return set_error(GIFT_EINVAL, "gift_ctx_profile_reset: ctx is NULL");
  gift_status st = drain_profile(ctx);
  if (st != GIFT_OK) return st;
  for (int k = 0; k < GIFT_KERNEL_COUNT; ++k) {
    ctx->prof_ms[k] = 0.0;
    ctx->prof_launches[k] = 0;
  }
  return GIFT_OK;
}

gift_status gift_factor_create(gift_ctx *ctx, int64_t m, int64_t n, int32_t rank, int32_t sides,
                               float damping, uint64_t seed, gift_factor **out) {
  if (!ctx || !out) return set_error(GIFT_EINVAL, "gift_factor_create: NULL argument");
  if (sides < GIFT_SIDE_INPUT || sides > GIFT_SIDE_BOTH)
    return set_error(GIFT_EINVAL, "gift_factor_create: sides must be INPUT, OUTPUT or BOTH");
  if (!(damping >= 0.f) || isinf(damping))
    return set_error(GIFT_EINVAL, "gift_factor_create: damping must be finite and >= 0");
  gift_status st = check_matrix_dims(m, n);
  if (st != GIFT_OK) return st;
  if (rank < 0 || rank > kMaxRank)
    return set_error(GIFT_ESHAPE, "gift_factor_create: rank must be in [0, 512]");
  if (side_in(sides, GIFT_SIDE_INPUT) && rank > n)
    return set_error(GIFT_ESHAPE, "gift_factor_create: rank exceeds n (input side)");
  if (side_in(sides, GIFT_SIDE_OUTPUT) && rank > m)
    return set_error(GIFT_ESHAPE, "gift_factor_create: rank exceeds m (output side)");
  if ((st = bind_device(ctx)) != GIFT_OK) return st;

  gift_factor *f = new (std::nothrow) gift_factor();
  if (!f) return set_error(GIFT_ENOMEM, "gift_factor_create: out of host memory");
  f->ctx = ctx;
  f->m = m;
  f->n = n;
  f->rank = rank;
  f->sides = sides;
  f->damping = damping;
  f->seed = seed;
  Side *list[2] = {&f->A, &f->G};
  const bool on[2] = {side_in(sides, GIFT_SIDE_INPUT), side_in(sides, GIFT_SIDE_OUTPUT)};
  const int64_t dims[2] = {n, m};
  size_t total = 0;
  for (int i = 0; i < 2; ++i) {
    Side &s = *list[i];
    s.dim = dims[i];
    s.r = on[i] ? rank : 0;
    s.k = (int32_t)(2 * (int64_t)s.r < s.dim ? 2 * s.r : s.dim);
    if (s.r == 0) continue;
    total += 4 * a256(sizeof(float) * s.dim * s.r) + 3 * a256(sizeof(float) * s.r) + a256(sizeof(float)) +
             a256(sizeof(float) * (size_t)s.k * s.dim);
  }
  if (total > 0) {
    hipError_t e = hipMalloc(&f->alloc, total);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      delete f;
      return set_error(GIFT_ENOMEM, "gift_factor_create: device allocation failed");
    }
    char *p = static_cast<char *>(f->alloc);
    for (int i = 0; i < 2; ++i) {
      Side &s = *list[i];
      if (s.r == 0) continue;
      auto take = [&](size_t bytes) {
        float *q = reinterpret_cast<float *>(p);
        p += a256(bytes);
        return q;
      };
      s.Ut = take(sizeof(float) * s.dim * s.r);
      s.U = take(sizeof(float) * s.dim * s.r);
      s.Uc = take(sizeof(float) * s.dim * s.r);
      s.Uci = take(sizeof(float) * s.dim * s.r);
      s.c_fwd = take(sizeof(float) * s.r);
      s.c_inv = take(sizeof(float) * s.r);
      s.lam = take(sizeof(float) * s.r);
      s.sigma2 = take(sizeof(float));
      s.Qt = take(sizeof(float) * (size_t)s.k * s.dim);
      if ((st = side_set_identity(ctx, s)) != GIFT_OK) {
        (void)hipFree(f->alloc);
        delete f;
        return st;
      }
    }
  }
  *out = f;
  return GIFT_OK;
}

gift_status gift_factor_create_chol(gift_ctx *ctx, int64_t m, int64_t n, int32_t block, int32_t sides,
                                    float damping, gift_factor **out) {
  if (!ctx || !out) return set_error(GIFT_EINVAL, "gift_factor_create_chol: NULL argument");
  if (sides < GIFT_SIDE_INPUT || sides > GIFT_SIDE_BOTH)
    return set_error(GIFT_EINVAL, "gift_factor_create_chol: sides must be INPUT, OUTPUT or BOTH");
  if (!(damping > 0.f) || isinf(damping))
    return set_error(GIFT_EINVAL, "gift_factor_create_chol: damping must be finite and > 0");
  gift_status st = check_matrix_dims(m, n);
  if (st != GIFT_OK) return st;
  if (block < 0) return set_error(GIFT_ESHAPE, "gift_factor_create_chol: block must be >= 0");
  const bool on[2] = {side_in(sides, GIFT_SIDE_INPUT), side_in(sides, GIFT_SIDE_OUTPUT)};
  const int64_t dims[2] = {n, m};
  int64_t beff[2] = {0, 0};
  for (int i = 0; i < 2; ++i) {
    if (!on[i]) continue;
    beff[i] = block == 0 || block >= dims[i] ? dims[i] : block;
    if (beff[i] > kMaxCholBlock)
      return set_error(GIFT_ESHAPE, "gift_factor_create_chol: block (or the full dim) exceeds 8192");
  }
  if ((st = bind_device(ctx)) != GIFT_OK) return st;
  gift_factor *f = new (std::nothrow) gift_factor();
  if (!f) return set_error(GIFT_ENOMEM, "gift_factor_create_chol: out of host memory");
  f->ctx = ctx;
  f->m = m;
  f->n = n;
  f->sides = sides;
  f->damping = damping;
  f->chol = true;
  f->block = block;
  f->A.dim = n;
  f->G.dim = m;
  CholSide *list[2] = {&f->CA, &f->CG};
  size_t total = 0;
  for (int i = 0; i < 2; ++i) {
    CholSide &s = *list[i];
    s.dim = dims[i];
    if (!on[i]) continue;
    s.b = (int32_t)beff[i];
    s.nblk = (int32_t)((dims[i] + beff[i] - 1) / beff[i]);
    const size_t blocks = (size_t)s.nblk * s.b * s.b;
    total += 2 * a256(sizeof(float) * blocks) + a256(sizeof(float) * (size_t)s.dim * s.dim) +
             a256(2 * sizeof(float));
  }
  hipError_t e = hipMalloc(&f->alloc, total);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    delete f;
    return set_error(GIFT_ENOMEM, "gift_factor_create_chol: device allocation failed");
  }
  char *p = static_cast<char *>(f->alloc);
  auto take = [&](size_t bytes) {
    float *q = reinterpret_cast<float *>(p);
    p += a256(bytes);
    return q;
  };
  for (int i = 0; i < 2; ++i) {
    CholSide &s = *list[i];
    if (s.b == 0) continue;
    const size_t blocks = (size_t)s.nblk * s.b * s.b;
    s.R = take(sizeof(float) * blocks);
    s.Rinv = take(sizeof(float) * blocks);
    s.A = take(sizeof(float) * (size_t)s.dim * s.dim);
    s.shift = take(2 * sizeof(float));
    if ((st = chol_side_identity(ctx, s)) != GIFT_OK) {
      (void)hipFree(f->alloc);
      delete f;
      return st;
    }
  }
  *out = f;
  return GIFT_OK;
}

void gift_factor_destroy(gift_factor *f) {
  if (!f) return;
  if (f->alloc) {
    (void)hipStreamSynchronize(f->ctx->stream);
    (void)hipFree(f->alloc);
  }
  delete f;
}

gift_status gift_statistics(gift_ctx *ctx, const void *x, int64_t T, int64_t dim, gift_dtype dtype,
                            float *A) {
  if (!ctx || !x || !A) return set_error(GIFT_EINVAL, "gift_statistics: NULL argument");
  if (dtype != GIFT_F32 && dtype != GIFT_BF16)
    return set_error(GIFT_EINVAL, "gift_statistics: dtype must be GIFT_F32 or GIFT_BF16");
  if (T <= 0 || dim <= 0) return set_error(GIFT_ESHAPE, "gift_statistics: T and dim must be positive");
  if (dim > kMaxRows) return set_error(GIFT_ESHAPE, "gift_statistics: dim exceeds the supported maximum (1048560)");
  gift_status st = bind_device(ctx);
  if (st != GIFT_OK) return st;
  const bool widen = dtype == GIFT_BF16 && !statistics_direct(dtype, dim);
  void *ws = nullptr;
  if ((st = workspace(ctx, widen ? sizeof(float) * (size_t)T * dim : 256, &ws)) != GIFT_OK) return st;
  float *Xc = widen ? static_cast<float *>(ws) : nullptr;
  void *d_tab = nullptr;
  if ((st = upload_table(ctx, TAB_STATS, nullptr, &x, sizeof(void *), &d_tab)) != GIFT_OK) return st;
  return launch_statistics(ctx, static_cast<const void *const *>(d_tab), &x, 1, T, dim, dtype, A, Xc);
}

gift_status gift_factor_update_batch(gift_ctx *ctx, int32_t count, gift_factor *const *factors,
                                     const void *const *acts, const void *const *out_grads,
                                     int64_t T, gift_dtype dtype, int32_t iters) {
  if (!ctx) return set_error(GIFT_EINVAL, "gift_factor_update: ctx is NULL");
  if (count < 0) return set_error(GIFT_EINVAL, "gift_factor_update: count must be >= 0");
  if (count > 0 && !factors) return set_error(GIFT_EINVAL, "gift_factor_update: factors is NULL");
  if (dtype != GIFT_F32 && dtype != GIFT_BF16)
    return set_error(GIFT_EINVAL, "gift_factor_update: dtype must be GIFT_F32 or GIFT_BF16");
  if (iters < 0) return set_error(GIFT_EINVAL, "gift_factor_update: iters must be >= 0");
  if (T <= 0) return set_error(GIFT_ESHAPE, "gift_factor_update: T must be positive");
  std::vector<SideJob> jobs;
  for (int32_t i = 0; i < count; ++i) {
    gift_factor *f = factors[i];
    if (!f) return set_error(GIFT_EINVAL, "gift_factor_update: NULL factor in the batch");
    for (int32_t j = 0; j < i; ++j)
      if (factors[j] == f) return set_error(GIFT_EINVAL, "gift_factor_update: a factor appears twice");
    const void *a = acts ? acts[i] : nullptr;
    const void *d = out_grads ? out_grads[i] : nullptr;
    if (f->chol) {
      if (f->CA.b > 0 && !a)
        return set_error(GIFT_EINVAL, "gift_factor_update: acts is NULL for an input-side factor");
      if (f->CG.b > 0 && !d)
        return set_error(GIFT_EINVAL, "gift_factor_update: out_grads is NULL for an output-side factor");
      continue;
    }
    if (f->A.r > 0) {
      if (!a) return set_error(GIFT_EINVAL, "gift_factor_update: acts is NULL for an input-side factor");
      jobs.push_back(SideJob{&f->A, a, f->seed, f->damping});
    }
    if (f->G.r > 0) {
      if (!d) return set_error(GIFT_EINVAL, "gift_factor_update: out_grads is NULL for an output-side factor");
      jobs.push_back(SideJob{&f->G, d, f->seed + 1, f->damping});
    }
  }
  bool any_chol = false;
  for (int32_t i = 0; i < count; ++i) any_chol = any_chol || factors[i]->chol;
  if (jobs.empty() && !any_chol) return GIFT_OK;
  gift_status st = bind_device(ctx);
  if (st != GIFT_OK) return st;
  if (!jobs.empty() && (st = factor_refresh_batch(ctx, jobs, T, dtype, iters)) != GIFT_OK) return st;
  for (int32_t i = 0; i < count; ++i) {
    gift_factor *f = factors[i];
    if (!f->chol) continue;
    if (f->CA.b > 0 && (st = chol_side_update(ctx, f->CA, acts[i], T, dtype, f->damping)) != GIFT_OK)
      return st;
    if (f->CG.b > 0 && (st = chol_side_update(ctx, f->CG, out_grads[i], T, dtype, f->damping)) != GIFT_OK)
      return st;
  }
  return GIFT_OK;
}

gift_status gift_factor_update(gift_ctx *ctx, gift_factor *f, const void *acts,
                               const void *out_grads, int64_t T, gift_dtype dtype, int32_t iters) {
  if (!ctx || !f) return set_error(GIFT_EINVAL, "gift_factor_update: NULL ctx or factor");
  return gift_factor_update_batch(ctx, 1, &f, &acts, &out_grads, T, dtype, iters);
}

static gift_status pick_side(const gift_factor *f, int32_t side, const Side **s) {
  if (side == GIFT_SIDE_INPUT) *s = &f->A;
  else if (side == GIFT_SIDE_OUTPUT) *s = &f->G;
  else return set_error(GIFT_EINVAL, "side must be GIFT_SIDE_INPUT or GIFT_SIDE_OUTPUT");
  if ((*s)->r == 0 && !side_in(f->sides, side))
    return set_error(GIFT_EINVAL, "the factor does not have this side");
  return GIFT_OK;
}

static gift_status pick_chol_side(const gift_factor *f, int32_t side, const CholSide **s) {
  if (!f->chol) return set_error(GIFT_EINVAL, "not a Cholesky-form factor");
  if (side == GIFT_SIDE_INPUT) *s = &f->CA;
  else if (side == GIFT_SIDE_OUTPUT) *s = &f->CG;
  else return set_error(GIFT_EINVAL, "side must be GIFT_SIDE_INPUT or GIFT_SIDE_OUTPUT");
  if ((*s)->b == 0) return set_error(GIFT_EINVAL, "the factor does not have this side");
  return GIFT_OK;
}

gift_status gift_factor_export_chol(gift_ctx *ctx, const gift_factor *f, int32_t side, float *R,
                                    float *Rinv) {
  if (!ctx || !f || !R || !Rinv) return set_error(GIFT_EINVAL, "gift_factor_export_chol: NULL argument");
  const CholSide *s = nullptr;
  gift_status st = pick_chol_side(f, side, &s);
  if (st != GIFT_OK) return st;
  if ((st = bind_device(ctx)) != GIFT_OK) return st;
  const size_t bytes = sizeof(float) * (size_t)s->nblk * s->b * s->b;
  GIFT_HIP_TRY(hipMemcpyAsync(R, s->R, bytes, hipMemcpyDeviceToDevice, ctx->stream));
  GIFT_HIP_TRY(hipMemcpyAsync(Rinv, s->Rinv, bytes, hipMemcpyDeviceToDevice, ctx->stream));
  return GIFT_OK;
}

gift_status gift_factor_import_chol(gift_ctx *ctx, gift_factor *f, int32_t side, const float *R,
                                    const float *Rinv) {
  if (!ctx || !f || !R || !Rinv) return set_error(GIFT_EINVAL, "gift_factor_import_chol: NULL argument");
  const CholSide *s = nullptr;
  gift_status st = pick_chol_side(f, side, &s);
  if (st != GIFT_OK) return st;
  if ((st = bind_device(ctx)) != GIFT_OK) return st;
  const size_t bytes = sizeof(float) * (size_t)s->nblk * s->b * s->b;
  GIFT_HIP_TRY(hipMemcpyAsync(s->R, R, bytes, hipMemcpyDeviceToDevice, ctx->stream));
  GIFT_HIP_TRY(hipMemcpyAsync(s->Rinv, Rinv, bytes, hipMemcpyDeviceToDevice, ctx->stream));
  return GIFT_OK;
}

gift_status gift_factor_export(gift_ctx *ctx, const gift_factor *f, int32_t side, float *U,
                               float *c_fwd, float *c_inv, float *sigma2) {
  if (!ctx || !f || !sigma2) return set_error(GIFT_EINVAL, "gift_factor_export: NULL argument");
  if (f->chol) return set_error(GIFT_EINVAL, "gift_factor_export: a Cholesky-form factor (use _chol)");
  const Side *s = nullptr;
  gift_status st = pick_side(f, side, &s);
  if (st != GIFT_OK) return st;
  if (s->r > 0 && (!U || !c_fwd || !c_inv))
    return set_error(GIFT_EINVAL, "gift_factor_export: NULL output");
  if ((st = bind_device(ctx)) != GIFT_OK) return st;
  return side_export(ctx, *s, U, c_fwd, c_inv, sigma2);
}

gift_status gift_factor_import(gift_ctx *ctx, gift_factor *f, int32_t side, const float *U,
                               const float *c_fwd, const float *c_inv, const float *sigma2) {
  if (!ctx || !f || !sigma2) return set_error(GIFT_EINVAL, "gift_factor_import: NULL argument");
  if (f->chol) return set_error(GIFT_EINVAL, "gift_factor_import: a Cholesky-form factor (use _chol)");
  const Side *cs = nullptr;
  gift_status st = pick_side(f, side, &cs);
  if (st != GIFT_OK) return st;
  Side *s = const_cast<Side *>(cs);
  if (s->r > 0 && (!U || !c_fwd || !c_inv))
    return set_error(GIFT_EINVAL, "gift_factor_import: NULL input");
  if ((st = bind_device(ctx)) != GIFT_OK) return st;
  return side_import(ctx, *s, U, c_fwd, c_inv, sigma2);
}

// Host-side checks shared by the encode entry points (no HIP call).
static gift_status encode_validate(gift_ctx *ctx, const gift_factor *f, const float *grads, int32_t N,
                                   int64_t m, int64_t n, int32_t block_rows, int32_t block_cols,
                                   gift_scale_mode mode, const uint8_t *codes, const float *scales) {
  if (!ctx) return set_error(GIFT_EINVAL, "gift_encode: ctx is NULL");
  if (!grads || !codes || !scales) return set_error(GIFT_EINVAL, "gift_encode: NULL tensor");
  if (mode != GIFT_SCALE_LOCAL && mode != GIFT_SCALE_SHARED)
    return set_error(GIFT_EINVAL, "gift_encode: unknown scale mode");
  if (N <= 0 || N > kMaxRanks) return set_error(GIFT_ESHAPE, "gift_encode: N must be in [1, 65535]");
  gift_status st = check_matrix_dims(m, n);
  if (st != GIFT_OK) return st;
  if (block_rows < 0 || block_cols < 0)
    return set_error(GIFT_ESHAPE, "gift_encode: block sizes must be >= 0");
  if (f && (f->m != m || f->n != n))
    return set_error(GIFT_ESHAPE, "gift_encode: factor was created for another shape");
  return GIFT_OK;
}

// A fixed device region that an allocation-free encode carves its scratch
// from (sub-slots, finalize buffer, projections, stored W~, Cholesky-form
// transform), instead of the context's grow-only buffers.
struct FixedScratch {
  char *base = nullptr;
  size_t cap = 0;
};

// Bytes of fixed scratch encode_impl carves for this call (mirrors its
// buffer plan; no HIP call).
static gift_status encode_fixed_bytes(gift_ctx *ctx, const gift_factor *f, const float *grads, int32_t N,
                                      int64_t m, int64_t n, int32_t block_rows, int32_t block_cols,
                                      const float *ef, const uint8_t *codes, const float *transformed,
                                      size_t *out) {
  if (f && f->chol) {
    const bool two = chol_transform_needs_tmp(f);
    const size_t xb = a256(sizeof(float) * (size_t)N * m * n * (two ? 2 : 1));
    size_t rest = 0;
    // the Euclidean encode of W~ (held 256-byte aligned in the scratch)
    gift_status st = encode_fixed_bytes(ctx, nullptr, grads, N, m, n, block_rows, block_cols, ef, codes,
                                        transformed, &rest);
    if (st != GIFT_OK) return st;
    *out = xb + rest;
    return GIFT_OK;
  }
  const BlockGeom g = block_geom(m, n, block_rows, block_cols);
  const int64_t nblk = (int64_t)g.nbr * g.nbc;
  const size_t raw_bytes = a256(sizeof(uint32_t) * (size_t)N * nblk * kAmaxSlots);
  const size_t fin_bytes = a256(sizeof(uint32_t) * (size_t)N * nblk);
  LowRankPlan plan;
  size_t proj_bytes = 0;
  if (f) {
    gift_status st = plan_low_rank(ctx, f, grads, N, m, n, false, nullptr, &proj_bytes, &plan);
    if (st != GIFT_OK) return st;
  }
  const bool gemm = f && plan.active;
  const bool recompute = gemm && encode_recomputes(f, n, grads, ef, codes, transformed);
  const bool store_wt = gemm && !recompute && n % 4 == 0 && g.bc % 4 == 0;
  const size_t wt_bytes = store_wt && !transformed ? a256(sizeof(float) * (size_t)N * m * n) : 0;
  *out = raw_bytes + fin_bytes + proj_bytes + wt_bytes;
  return GIFT_OK;
}

static gift_status encode_impl(gift_ctx *ctx, const gift_factor *f, const float *grads, int32_t N,
                               int64_t m, int64_t n, int32_t block_rows, int32_t block_cols,
                               gift_scale_mode mode, float *ef, uint8_t *codes, float *scales,
                               float *transformed, uint32_t *hits, const FixedScratch *fx) {
  gift_status st = encode_validate(ctx, f, grads, N, m, n, block_rows, block_cols, mode, codes, scales);
  if (st != GIFT_OK) return st;
  if ((st = bind_device(ctx)) != GIFT_OK) return st;
  if (f && f->chol) {
    // W~ = L_G^-1 W L_A^-T into the transform buffer, then the Euclidean
    // encode of W~ (whose own workspace holds everything else)
    const size_t total = (size_t)N * m * n;
    const bool two = chol_transform_needs_tmp(f);
    const size_t xbytes = sizeof(float) * total * (two ? 2 : 1);
    void *buf = nullptr;
    FixedScratch rest;
    if (fx) {
      if (a256(xbytes) > fx->cap) return set_error(GIFT_ESHAPE, "gift_encode: fixed scratch too small");
      buf = fx->base;
      rest.base = fx->base + a256(xbytes);
      rest.cap = fx->cap - a256(xbytes);
    } else if ((st = grow_buffer(ctx, ctx->xform, xbytes, &buf)) != GIFT_OK) {
      return st;
    }
    float *wt = static_cast<float *>(buf);
    if ((st = launch_chol_transform(ctx, f, grads, wt, N, false, two ? wt + total : nullptr)) != GIFT_OK)
      return st;
    return encode_impl(ctx, nullptr, wt, N, m, n, block_rows, block_cols, mode, ef, codes, scales, transformed,
                       hits, fx ? &rest : nullptr);
  }
  const BlockGeom g = block_geom(m, n, block_rows, block_cols);
  const int64_t nblk = (int64_t)g.nbr * g.nbc;
  const size_t fin_bytes = a256(sizeof(uint32_t) * (size_t)N * nblk);
  LowRankPlan plan;
  size_t proj_bytes = 0;
  if (f && (st = plan_low_rank(ctx, f, grads, N, m, n, false, nullptr, &proj_bytes, &plan)) != GIFT_OK)
    return st;
  // With a transform, the AMAX pass computes W~ (+ R) for the block maxima and
  // the QUANT pass computes it again (same kernel arithmetic, so the same
  // values) when the split-bf16 kernels take the job; otherwise the AMAX pass
  // stores W~ (scratch unless the caller asked for it) and the QUANT pass
  // streams it.
  const bool gemm = f && plan.active;
  const bool recompute = gemm && encode_recomputes(f, n, grads, ef, codes, transformed);
  const bool store_wt = gemm && !recompute && n % 4 == 0 && g.bc % 4 == 0;
  const size_t wt_bytes = store_wt && !transformed ? a256(sizeof(float) * (size_t)N * m * n) : 0;
  const size_t raw_words = (size_t)N * nblk * kAmaxSlots;
  uint32_t *amax_raw = nullptr, *prev_set = nullptr;
  size_t prev_dirty = 0;
  void *ws = nullptr;
  if (fx) {
    // the fixed region holds the sub-slots (cleared here: the last call on
    // this device left its maxima in them), then the rest
    const size_t raw_bytes = a256(sizeof(uint32_t) * raw_words);
    if (raw_bytes + fin_bytes + proj_bytes + wt_bytes > fx->cap)
      return set_error(GIFT_ESHAPE, "gift_encode: fixed scratch too small");
    amax_raw = reinterpret_cast<uint32_t *>(fx->base);
    ws = fx->base + raw_bytes;
    if ((st = launch_zero_u32(ctx, amax_raw, (int64_t)raw_words)) != GIFT_OK) return st;
  } else {
    if ((st = amax_slots(ctx, raw_words, &amax_raw, &prev_set, &prev_dirty)) != GIFT_OK) return st;
    if ((st = workspace(ctx, fin_bytes + proj_bytes + wt_bytes, &ws)) != GIFT_OK) return st;
  }
  // book-keeping of the context's alternating sub-slot sets (not used by a
  // fixed region, which is cleared at the start of every call)
  auto slots_done = [&](size_t left) {
    if (!fx) amax_slots_done(ctx, left);
  };
  uint32_t *amax_fin = static_cast<uint32_t *>(ws);
  float *wt = transformed;
  if (wt_bytes) wt = reinterpret_cast<float *>(static_cast<char *>(ws) + fin_bytes + proj_bytes);
  TileJob job;
  if (gemm) {
    if ((st = plan_low_rank(ctx, f, grads, N, m, n, false, static_cast<char *>(ws) + fin_bytes, &proj_bytes,
                            &plan)) != GIFT_OK)
      return st;
    job = plan.upd;
  }
  job.M = m;
  job.N = n;
  job.batch = N;
  job.D = grads;
  job.ldd = n;
  job.dbs = m * n;
  job.amax = amax_raw;
  job.geom = g;
  job.shared = mode == GIFT_SCALE_SHARED;
  job.ef = ef;
  job.scales = scales;
  job.transformed = gemm ? wt : transformed;
  job.sweep_store = gemm && !recompute;
  job.kernel_family = gemm ? GIFT_KERNEL_UPDATE_AMAX : GIFT_KERNEL_AMAX;
  // both passes must take the same kernel, or their W~ would differ
  if (recompute && !lr_update_eligible(job))
    return set_error(GIFT_EUNSUPPORTED, "gift_encode: internal: split-bf16 update not applicable");
  if ((st = launch_tile(ctx, job)) != GIFT_OK) return st;
  job.transformed = nullptr;
  job.codes = codes;
  job.hits = hits;   // every quantize route counts the boundary hits as it packs
  // QUANT pass: the streaming kernel reads the raw sub-slots itself (on the
  // stored W~ + R with a transform, on W without); otherwise a finalize
  // launch reduces them first
  if (recompute && lr_quant_reads_raw(job)) {
    // the quantize pass reduces the raw sub-slots itself and writes the scales
    TileJob q = job;
    q.from_raw = true;
    q.clear = prev_set;
    q.clear_words = (int64_t)prev_dirty;
    q.kernel_family = GIFT_KERNEL_UPDATE_QUANT;
    if ((st = launch_tile(ctx, q)) != GIFT_OK) return st;
    slots_done(raw_words);
    return GIFT_OK;
  }
  const float *qsrc = gemm ? wt : grads;
  if (!recompute && qsrc && stream_eligible(m, n, g, qsrc, codes, ef, nullptr)) {
    TileJob q = job;
    q.nseg = 0;
    q.D = qsrc;
    q.ef_added = gemm;
    q.from_raw = true;
    q.clear = prev_set;
    q.clear_words = (int64_t)prev_dirty;
    q.kernel_family = gemm ? GIFT_KERNEL_UPDATE_QUANT : GIFT_KERNEL_QUANT;
    if ((st = launch_stream_codec(ctx, q)) != GIFT_OK) return st;
    slots_done(raw_words);
    return GIFT_OK;
  }
  if ((st = launch_finalize_amax(ctx, amax_raw, N, nblk, job.shared, amax_fin, scales, prev_set,
                                 (int64_t)prev_dirty)) != GIFT_OK)
    return st;
  job.amax = amax_fin;
  job.kernel_family = gemm ? GIFT_KERNEL_UPDATE_QUANT : GIFT_KERNEL_QUANT;
  if ((st = launch_tile(ctx, job)) != GIFT_OK) return st;
  slots_done(0);
  return GIFT_OK;
}

namespace {
// Device address of this device's `scratch` array, looked up once per device
// (hipGetSymbolAddress with the device current) and kept.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

gift_status noalloc_scratch(gift_ctx *ctx, char **out) {
  int dev = -1;
  GIFT_HIP_TRY(hipGetDevice(&dev));
  if (dev != ctx->device)
    return set_error(GIFT_EINVAL, "gift_encode_noalloc: the context's device must be the current device");
  if (dev < 0 || dev >= kMaxDevices)
    return set_error(GIFT_EUNSUPPORTED, "gift_encode_noalloc: device index above 63");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_error(e, "gift_encode_noalloc: hipGetSymbolAddress(scratch)");
    if (!p) return set_error(GIFT_EHIP, "gift_encode_noalloc: no device address for the scratch array");
    g_scratch_ptr[dev] = p;
  }
  *out = static_cast<char *>(g_scratch_ptr[dev]);
  return GIFT_OK;
}

// Marks the context for the duration of an allocation-free call (no
// profiling events are created or recorded).
struct NoAllocCall {
  gift_ctx *ctx;
  explicit NoAllocCall(gift_ctx *c) : ctx(c) { ctx->no_alloc_call = true; }
  ~NoAllocCall() { ctx->no_alloc_call = false; }
};
}  // namespace

gift_status gift_encode(gift_ctx *ctx, const gift_factor *f, const float *grads, int32_t N,
                        int64_t m, int64_t n, int32_t block_rows, int32_t block_cols,
                        gift_scale_mode mode, float *ef, uint8_t *codes, float *scales,
                        float *transformed) {
  return encode_impl(ctx, f, grads, N, m, n, block_rows, block_cols, mode, ef, codes, scales, transformed,
                     nullptr, nullptr);
}

gift_status gift_encode_noalloc(gift_ctx *ctx, const gift_factor *f, const float *grads, int32_t N,
                                int64_t m, int64_t n, int32_t block_rows, int32_t block_cols,
                                gift_scale_mode mode, float *ef, uint8_t *codes, float *scales,
                                float *transformed) {
  gift_status st = encode_validate(ctx, f, grads, N, m, n, block_rows, block_cols, mode, codes, scales);
  if (st != GIFT_OK) return st;
  size_t need = 0;
  if ((st = encode_fixed_bytes(ctx, f, grads, N, m, n, block_rows, block_cols, ef, codes, transformed,
                               &need)) != GIFT_OK)
    return st;
  if (need > (size_t)GIFT_NOALLOC_SCRATCH_BYTES)
    return set_error(GIFT_ESHAPE, "gift_encode_noalloc: this encode needs " + std::to_string(need) +
                                      " bytes of scratch, more than the fixed " +
                                      std::to_string((size_t)GIFT_NOALLOC_SCRATCH_BYTES) +
                                      " (split the call into fewer ranks or rows, or pass `transformed`)");
  if ((st = bind_device(ctx)) != GIFT_OK) return st;
  FixedScratch fx;
  if ((st = noalloc_scratch(ctx, &fx.base)) != GIFT_OK) return st;
  fx.cap = (size_t)GIFT_NOALLOC_SCRATCH_BYTES;
  NoAllocCall mark(ctx);
  return encode_impl(ctx, f, grads, N, m, n, block_rows, block_cols, mode, ef, codes, scales, transformed,
                     nullptr, &fx);
}

gift_status gift_encode_hits(gift_ctx *ctx, const gift_factor *f, const float *grads, int32_t N,
                             int64_t m, int64_t n, int32_t block_rows, int32_t block_cols,
                             gift_scale_mode mode, float *ef, uint8_t *codes, float *scales,
                             float *transformed, uint32_t *hits) {
  if (!hits) return set_error(GIFT_EINVAL, "gift_encode_hits: hits is NULL");
  if (reinterpret_cast<uintptr_t>(hits) & 3)
    return set_error(GIFT_EINVAL, "gift_encode_hits: hits must be 4-byte aligned");
  return encode_impl(ctx, f, grads, N, m, n, block_rows, block_cols, mode, ef, codes, scales, transformed,
                     hits, nullptr);
}

gift_status gift_reduce_local(gift_ctx *ctx, const uint8_t *codes, const float *scales, int32_t N,
                              int64_t m, int64_t n, int32_t block_rows, int32_t block_cols,
                              float *mean) {
  if (!ctx) return set_error(GIFT_EINVAL, "gift_reduce_local: ctx is NULL");
  if (!codes || !scales || !mean) return set_error(GIFT_EINVAL, "gift_reduce_local: NULL tensor");
  if (N <= 0 || N > kMaxRanks)
    return set_error(GIFT_ESHAPE, "gift_reduce_local: N must be in [1, 65535]");
  gift_status st = check_matrix_dims(m, n);
  if (st != GIFT_OK) return st;
  if (block_rows < 0 || block_cols < 0)
    return set_error(GIFT_ESHAPE, "gift_reduce_local: block sizes must be >= 0");
  if ((st = bind_device(ctx)) != GIFT_OK) return st;
  return launch_reduce(ctx, codes, scales, N, m, n, block_geom(m, n, block_rows, block_cols), mean);
}

gift_status gift_encode_mxfp4(gift_ctx *ctx, const gift_factor *f, const float *grads, int32_t N,
                              int64_t m, int64_t n, float *ef, uint8_t *codes, uint8_t *scales,
                              float *transformed) {
  if (!ctx) return set_error(GIFT_EINVAL, "gift_encode_mxfp4: ctx is NULL");
  if (!grads || !codes || !scales) return set_error(GIFT_EINVAL, "gift_encode_mxfp4: NULL tensor");
  if (N <= 0 || N > kMaxRanks) return set_error(GIFT_ESHAPE, "gift_encode_mxfp4: N must be in [1, 65535]");
  gift_status st = check_matrix_dims(m, n);
  if (st != GIFT_OK) return st;
  if (n % 32 != 0) return set_error(GIFT_ESHAPE, "gift_encode_mxfp4: n must be a multiple of 32");
  if (f && (f->m != m || f->n != n))
    return set_error(GIFT_ESHAPE, "gift_encode_mxfp4: factor was created for another shape");
  if (!al16p(grads) || (ef && !al16p(ef)) || (transformed && !al16p(transformed)) ||
      (reinterpret_cast<uintptr_t>(codes) & 3))
    return set_error(GIFT_EINVAL,
                     "gift_encode_mxfp4: grads, ef and transformed must be 16-byte aligned, codes 4-byte aligned");
  if ((st = bind_device(ctx)) != GIFT_OK) return st;
  const int64_t total = (int64_t)N * m * n;
  const float *src = grads;
  if (f) {
    if (f->chol) {
      const bool two = chol_transform_needs_tmp(f);
      void *buf = nullptr;
      if ((st = grow_buffer(ctx, ctx->xform, sizeof(float) * (size_t)total * (two ? 2 : 1), &buf)) != GIFT_OK)
        return st;
      float *wt = static_cast<float *>(buf);
      if ((st = launch_chol_transform(ctx, f, grads, wt, N, false, two ? wt + total : nullptr)) != GIFT_OK)
        return st;
      src = wt;
    } else {
      LowRankPlan plan;
      size_t bytes = 0;
      if ((st = plan_low_rank(ctx, f, grads, N, m, n, false, nullptr, &bytes, &plan)) != GIFT_OK) return st;
      if (plan.active) {
        void *ws = nullptr;
        if ((st = workspace(ctx, bytes, &ws)) != GIFT_OK) return st;
        if ((st = plan_low_rank(ctx, f, grads, N, m, n, false, static_cast<char *>(ws), &bytes, &plan)) !=
            GIFT_OK)
          return st;
        // the split-bf16 update computes W~ (+ R) and packs MXFP4 in one pass
        TileJob mj = plan.upd;
        mj.D = grads;
        mj.ldd = n;
        mj.dbs = m * n;
        mj.ef = ef;
        mj.transformed = transformed;
        mj.mx_codes = codes;
        mj.mx_scales = scales;
        mj.kernel_family = GIFT_KERNEL_MXFP4;
        if (lr_update_eligible(mj)) return launch_lr_update(ctx, mj);
        void *buf = nullptr;
        if ((st = grow_buffer(ctx, ctx->xform, sizeof(float) * (size_t)total, &buf)) != GIFT_OK) return st;
        // W~ = W + the low-rank part, stored (float32 products)
        TileJob job = plan.upd;
        job.C = static_cast<float *>(buf);
        job.ldc = n;
        job.cbs = m * n;
        job.D = grads;
        job.ldd = n;
        job.dbs = m * n;
        job.beta = 1.f;
        job.split3 = false;
        job.kernel_family = GIFT_KERNEL_UPDATE_STORE;
        if ((st = launch_tile(ctx, job)) != GIFT_OK) return st;
        src = static_cast<float *>(buf);
      }
    }
  }
  return launch_mx_quant(ctx, src, ef, ef, transformed, codes, scales, total);
}

gift_status gift_reduce_local_mxfp4(gift_ctx *ctx, const uint8_t *codes, const uint8_t *scales, int32_t N,
                                    int64_t m, int64_t n, float *mean) {
  if (!ctx) return set_error(GIFT_EINVAL, "gift_reduce_local_mxfp4: ctx is NULL");
  if (!codes || !scales || !mean) return set_error(GIFT_EINVAL, "gift_reduce_local_mxfp4: NULL tensor");
  if (N <= 0 || N > kMaxRanks)
    return set_error(GIFT_ESHAPE, "gift_reduce_local_mxfp4: N must be in [1, 65535]");
  gift_status st = check_matrix_dims(m, n);
  if (st != GIFT_OK) return st;
  if (n % 32 != 0) return set_error(GIFT_ESHAPE, "gift_reduce_local_mxfp4: n must be a multiple of 32");
  if ((reinterpret_cast<uintptr_t>(codes) & 3) || !al16p(mean))
    return set_error(GIFT_EINVAL, "gift_reduce_local_mxfp4: codes must be 4-byte, mean 16-byte aligned");
  if ((st = bind_device(ctx)) != GIFT_OK) return st;
  return launch_mx_reduce(ctx, codes, scales, N, m * n, mean);
}

gift_status gift_decode(gift_ctx *ctx, const gift_factor *f, const float *mean, int64_t m,
                        int64_t n, float *out) {
  if (!ctx) return set_error(GIFT_EINVAL, "gift_decode: ctx is NULL");
  if (!mean || !out) return set_error(GIFT_EINVAL, "gift_decode: NULL tensor");
  if (mean == out) return set_error(GIFT_EINVAL, "gift_decode: out must not alias mean");
  gift_status st = check_matrix_dims(m, n);
  if (st != GIFT_OK) return st;
  if (f && (f->m != m || f->n != n))
    return set_error(GIFT_ESHAPE, "gift_decode: factor was created for another shape");
  if ((st = bind_device(ctx)) != GIFT_OK) return st;
  if (f && f->chol) {
    float *tmp = nullptr;
    if (chol_transform_needs_tmp(f)) {
      void *buf = nullptr;
      if ((st = grow_buffer(ctx, ctx->xform, sizeof(float) * (size_t)m * n, &buf)) != GIFT_OK) return st;
      tmp = static_cast<float *>(buf);
    }
    return launch_chol_transform(ctx, f, mean, out, 1, true, tmp);
  }
  LowRankPlan plan;
  size_t bytes = 0;
  if (f && (st = plan_low_rank(ctx, f, mean, 1, m, n, true, nullptr, &bytes, &plan)) != GIFT_OK)
    return st;
  if (!plan.active) return launch_copy_f32(ctx, out, mean, m * n);
  void *ws = nullptr;
  if ((st = workspace(ctx, bytes, &ws)) != GIFT_OK) return st;
  if ((st = plan_low_rank(ctx, f, mean, 1, m, n, true, static_cast<char *>(ws), &bytes, &plan)) != GIFT_OK)
    return st;
  TileJob job = plan.upd;
  job.C = out;
  job.ldc = n;
  job.cbs = m * n;
  job.D = mean;
  job.ldd = n;
  job.dbs = m * n;
  job.beta = 1.f;
  job.kernel_family = GIFT_KERNEL_UPDATE_STORE;
  return launch_tile(ctx, job);
}

// gift_decode_batch for two-sided low-rank factors of one rank r (both
// sides, 16 to 128): one launch per product over all matrices, each
// matrix's mean, output and factor operands reached through device pointer
// tables; every product takes the kernel, split-K partials and summation
// order that gift_decode takes for one matrix (eq. design_full_inverse_transform:
// P = M U_A, Q = U_G^T M, K = U_G^T P, L2 = (P + U_G C'_G K) C'_A, then
// out = M + (U_G C'_G) Q + L2 U_A^T), so the outputs equal its bit for bit.
// Returns GIFT_EUNSUPPORTED (nothing enqueued) when the shapes do not allow it.
static gift_status decode_batch_both(gift_ctx *ctx, int32_t count, const gift_factor *const *factors,
                                     const float *const *means, float *const *outs, int64_t m, int64_t n) {
  const gift_factor *f0 = factors[0];
  const int32_t r = f0->A.r;
  if (count < 2 || !(r == 16 || r == 32 || r == 64 || r == 128) || f0->G.r != r || n % 4 != 0 ||
      m * n >= (1LL << 29))
    return GIFT_EUNSUPPORTED;
  for (int32_t i = 0; i < count; ++i) {
    const gift_factor *f = factors[i];
    if (!f || f->chol || !side_in(f->sides, GIFT_SIDE_INPUT) || !side_in(f->sides, GIFT_SIDE_OUTPUT) ||
        f->A.r != r || f->G.r != r || !al16p(means[i]) || !al16p(outs[i]) || !al16p(f->A.Ut) ||
        !al16p(f->A.U) || !al16p(f->A.c_inv) || !al16p(f->G.Ut) || !al16p(f->G.Uci))
      return GIFT_EUNSUPPORTED;
  }
  // gift_decode's partial counts for one matrix
  const int pparts = proj_parts(m, n, r, 1);
  const bool presum = pparts > 1;
  const int qsplit = (n * r) % 4 == 0 ? small_split(n, r, 1, m) : 1;
  const int ksplit = ((int64_t)r * r) % 4 == 0 ? small_split(r, r, 1, m) : 1;
  TileJob pj;
  pj.nseg = 1;
  pj.seg[0].a = Operand{means[0], n, 0, true};
  pj.seg[0].b = Operand{f0->A.Ut, n, 0, true};
  pj.seg[0].K = n;
  pj.M = m;
  pj.N = r;
  pj.batch = count;
  pj.ldc = r;
  pj.cbs = m * r;
  pj.ksplit = pparts;
  pj.kernel_family = GIFT_KERNEL_DECODE_PROJECT;
  // workspace: P (partials), its sum, Q (partials), K (partials), L2
  const int64_t C = count;
  size_t off = 0;
  auto carve = [&](size_t floats) {
    const size_t at = off;
    off += a256(sizeof(float) * floats);
    return at;
  };
  const size_t oP = carve((size_t)C * pparts * m * r), oPs = presum ? carve((size_t)C * m * r) : 0;
  const size_t oQ = carve((size_t)C * n * r), oQp = qsplit > 1 ? carve((size_t)C * qsplit * n * r) : 0;
  const size_t oK = carve((size_t)C * r * r), oKp = ksplit > 1 ? carve((size_t)C * ksplit * r * r) : 0;
  const size_t oL = carve((size_t)C * m * r);
  void *ws = nullptr;
  gift_status st;
  if ((st = workspace(ctx, off, &ws)) != GIFT_OK) return st;
  char *w = static_cast<char *>(ws);
  float *P = reinterpret_cast<float *>(w + oP), *Ps = presum ? reinterpret_cast<float *>(w + oPs) : P;
  float *Qm = reinterpret_cast<float *>(w + oQ), *Qp = reinterpret_cast<float *>(w + oQp);
  float *Km = reinterpret_cast<float *>(w + oK), *Kp = reinterpret_cast<float *>(w + oKp);
  float *L2 = reinterpret_cast<float *>(w + oL);
  // device tables: means, outputs, U_G^T, U_G diag(c'_G), U_A, c'_A per matrix
  std::vector<const void *> host((size_t)6 * count);
  for (int32_t i = 0; i < count; ++i) {
    host[0 * (size_t)count + i] = means[i];
    host[1 * (size_t)count + i] = outs[i];
    host[2 * (size_t)count + i] = factors[i]->G.Ut;
    host[3 * (size_t)count + i] = factors[i]->G.Uci;
    host[4 * (size_t)count + i] = factors[i]->A.U;
    host[5 * (size_t)count + i] = factors[i]->A.c_inv;
  }
  void *tb = nullptr;
  if ((st = upload_table(ctx, TAB_DECODE_BOTH, f0, host.data(), sizeof(void *) * host.size(), &tb)) != GIFT_OK)
    return st;
  const float *const *t_mean = static_cast<const float *const *>(tb);
  float *const *t_out = const_cast<float *const *>(t_mean + count);
  const float *const *t_gut = t_mean + 2 * count, *const *t_guci = t_mean + 3 * count;
  const float *const *t_au = t_mean + 4 * count, *const *t_acinv = t_mean + 5 * count;
  std::vector<DecodePtrs> dp(count);
  for (int32_t i = 0; i < count; ++i) dp[i] = DecodePtrs{means[i], factors[i]->A.Ut, factors[i]->A.Uci, outs[i]};
  void *dt = nullptr;
  if ((st = upload_table(ctx, TAB_DECODE, f0, dp.data(), sizeof(DecodePtrs) * (size_t)count, &dt)) != GIFT_OK)
    return st;
  pj.C = P;
  pj.decode_tab = static_cast<const DecodePtrs *>(dt);
  // the final update on the register-direct kernel, as gift_decode's:
  // out = M + (U_G C'_G) Q + L2 U_A^T
  TileJob uj;
  uj.nseg = 2;
  uj.seg[0].a = Operand{nullptr, r, 0, true};
  uj.seg[0].a.tab = t_guci;
  uj.seg[0].b = Operand{Qm, r, n * r, true};
  uj.seg[0].K = r;
  uj.seg[1].a = Operand{L2, r, m * r, true};
  uj.seg[1].b = Operand{nullptr, r, 0, true};
  uj.seg[1].b.tab = t_au;
  uj.seg[1].K = r;
  uj.M = m;
  uj.N = n;
  uj.batch = count;
  uj.d_tab = t_mean;
  uj.c_tab = t_out;
  uj.ldc = n;
  uj.cbs = m * n;
  uj.ldd = n;
  uj.dbs = m * n;
  uj.beta = 1.f;
  uj.kernel_family = GIFT_KERNEL_UPDATE_STORE;
  // both ends on the kernels gift_decode takes, or nothing is enqueued (the
  // tables and workspace stay for later calls)
  if (!proj_staged_eligible(pj) || !update_kernel_eligible(uj)) return GIFT_EUNSUPPORTED;
  // P = M U_A (partials, summed in order)
  if ((st = launch_proj(ctx, pj)) != GIFT_OK) return st;
  if (presum && (st = launch_lr_psum(ctx, P, Ps, pparts, m * r, count, GIFT_KERNEL_DECODE_PROJECT)) != GIFT_OK)
    return st;
  {  // Q^T = M^T U_G
    TileJob j;
    j.nseg = 1;
    j.seg[0].a = Operand{nullptr, n, m * n, false};
    j.seg[0].a.tab = t_mean;
    j.seg[0].b = Operand{nullptr, m, 0, true};
    j.seg[0].b.tab = t_gut;
    j.seg[0].K = m;
    j.M = n;
    j.N = r;
    j.batch = count;
    j.C = qsplit > 1 ? Qp : Qm;
    j.ldc = r;
    j.cbs = n * r;
    j.ksplit = qsplit;
    j.kernel_family = GIFT_KERNEL_DECODE_PROJECT;
    if ((st = launch_tile(ctx, j)) != GIFT_OK) return st;
    if (qsplit > 1 && (st = launch_lr_psum(ctx, Qp, Qm, qsplit, n * r, count, j.kernel_family)) != GIFT_OK)
      return st;
  }
  {  // K = U_G^T P
    TileJob j;
    j.nseg = 1;
    j.seg[0].a = Operand{nullptr, m, 0, true};
    j.seg[0].a.tab = t_gut;
    j.seg[0].b = Operand{Ps, r, m * r, false};
    j.seg[0].K = m;
    j.M = r;
    j.N = r;
    j.batch = count;
    j.C = ksplit > 1 ? Kp : Km;
    j.ldc = r;
    j.cbs = (int64_t)r * r;
    j.ksplit = ksplit;
    j.kernel_family = GIFT_KERNEL_DECODE_PROJECT;
    if ((st = launch_tile(ctx, j)) != GIFT_OK) return st;
    if (ksplit > 1 && (st = launch_lr_psum(ctx, Kp, Km, ksplit, (int64_t)r * r, count, j.kernel_family)) != GIFT_OK)
      return st;
  }
  {  // L2 = (P + U_G C'_G K) C'_A
    TileJob j;
    j.nseg = 1;
    j.seg[0].a = Operand{nullptr, r, 0, true};
    j.seg[0].a.tab = t_guci;
    j.seg[0].b = Operand{Km, r, (int64_t)r * r, false};
    j.seg[0].K = r;
    j.M = m;
    j.N = r;
    j.batch = count;
    j.C = L2;
    j.ldc = r;
    j.cbs = m * r;
    j.D = Ps;
    j.ldd = r;
    j.dbs = m * r;
    j.beta = 1.f;
    j.colscale_tab = t_acinv;
    j.kernel_family = GIFT_KERNEL_DECODE_PROJECT;
    if ((st = launch_tile(ctx, j)) != GIFT_OK) return st;
  }
  return launch_tile(ctx, uj);
}

gift_status gift_decode_batch(gift_ctx *ctx, int32_t count, const gift_factor *const *factors,
                              const float *const *means, float *const *outs, int64_t m, int64_t n) {
  if (!ctx) return set_error(GIFT_EINVAL, "gift_decode_batch: ctx is NULL");
  if (count < 0 || count > kMaxRanks)
    return set_error(GIFT_EINVAL, "gift_decode_batch: count must be in [0, 65535]");
  if (count == 0) return GIFT_OK;
  if (!factors || !means || !outs) return set_error(GIFT_EINVAL, "gift_decode_batch: NULL array");
  gift_status st = check_matrix_dims(m, n);
  if (st != GIFT_OK) return st;
  for (int32_t i = 0; i < count; ++i) {
    if (!means[i] || !outs[i]) return set_error(GIFT_EINVAL, "gift_decode_batch: NULL tensor");
    if (means[i] == outs[i]) return set_error(GIFT_EINVAL, "gift_decode_batch: out must not alias mean");
    if (factors[i] && (factors[i]->m != m || factors[i]->n != n))
      return set_error(GIFT_ESHAPE, "gift_decode_batch: factor was created for another shape");
    for (int32_t j = 0; j < i; ++j)
      if (outs[j] == outs[i]) return set_error(GIFT_EINVAL, "gift_decode_batch: an output appears twice");
  }
  if ((st = bind_device(ctx)) != GIFT_OK) return st;
  const gift_factor *f0 = factors[0];
  if (count > 1 && f0 && !f0->chol && f0->A.r > 0 && f0->G.r > 0) {
    st = decode_batch_both(ctx, count, factors, means, outs, m, n);
    if (st != GIFT_EUNSUPPORTED) return st;
  }
  // one launch per pass for input-side low-rank factors of one rank: the
  // kernels, split-K partials and summation order of gift_decode, with the
  // batch index running over the matrices
  bool grouped = count > 1 && f0 && !f0->chol && f0->A.r > 0 && f0->G.r == 0 && n % 4 == 0 &&
                 m * n < (1LL << 29);
  const int32_t r = grouped ? f0->A.r : 0;
  if (grouped && r != 16 && r != 32 && r != 64 && r != 128) grouped = false;
  for (int32_t i = 0; grouped && i < count; ++i) {
    const gift_factor *f = factors[i];
    grouped = f && !f->chol && f->A.r == r && f->G.r == 0 && al16p(means[i]) && al16p(outs[i]);
  }
  TileJob pj, uj;
  int pparts = 1;
  if (grouped) {
    pparts = proj_parts(m, n, r, 1);
    pj.nseg = 1;
    pj.seg[0].a = Operand{means[0], n, 0, true};
    pj.seg[0].b = Operand{f0->A.Ut, n, 0, true};
    pj.seg[0].K = n;
    pj.M = m;
    pj.N = r;
    pj.batch = count;
    pj.ldc = r;
    pj.cbs = m * r;
    pj.ksplit = pparts;
    pj.kernel_family = GIFT_KERNEL_DECODE_PROJECT;
    grouped = proj_staged_eligible(pj);
  }
  if (!grouped) {
    for (int32_t i = 0; i < count; ++i)
      if ((st = gift_decode(ctx, factors[i], means[i], m, n, outs[i])) != GIFT_OK) return st;
    return GIFT_OK;
  }
  void *ws = nullptr;
  if ((st = workspace(ctx, sizeof(float) * (size_t)count * pparts * m * r, &ws)) != GIFT_OK) return st;
  float *P = static_cast<float *>(ws);
  std::vector<DecodePtrs> host(count);
  for (int32_t i = 0; i < count; ++i)
    host[i] = DecodePtrs{means[i], factors[i]->A.Ut, factors[i]->A.Uci, outs[i]};
  void *tab = nullptr;
  if ((st = upload_table(ctx, TAB_DECODE, f0, host.data(), sizeof(DecodePtrs) * (size_t)count, &tab)) != GIFT_OK)
    return st;
  const DecodePtrs *d_tab = static_cast<const DecodePtrs *>(tab);
  pj.C = P;
  pj.decode_tab = d_tab;
  if ((st = launch_proj(ctx, pj)) != GIFT_OK) return st;
  uj.nseg = 1;
  uj.seg[0].a = Operand{P, r, m * r, true, pparts};
  uj.seg[0].b = Operand{f0->A.Uci, r, 0, true};
  uj.seg[0].K = r;
  uj.M = m;
  uj.N = n;
  uj.batch = count;
  uj.C = outs[0];
  uj.ldc = n;
  uj.cbs = m * n;
  uj.D = means[0];
  uj.ldd = n;
  uj.dbs = m * n;
  uj.beta = 1.f;
  uj.kernel_family = GIFT_KERNEL_UPDATE_STORE;
  uj.decode_tab = d_tab;
  if (!update_kernel_eligible(uj))
    return set_error(GIFT_EUNSUPPORTED, "gift_decode_batch: internal: update kernel not applicable");
  return launch_update(ctx, uj);
}

}  // extern "C"
