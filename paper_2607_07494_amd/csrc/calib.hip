// Peak calibration kernels for the benchmark's roofline (not part of the
// codec): matrix-core loops with no memory traffic, whose rate is the
// achievable dense MFMA throughput of this GPU for the two instruction kinds
// the codec uses (bf16 16x16x32 for the statistics and the split-bf16
// transforms, float32 16x16x4 for the inverse transform) and for their
// 32 x 32 output forms (bf16 32x32x16, float32 32x32x2), and a streaming
// read, the achievable HBM read rate (the encode is almost all reads).
// Built into libgift_calib.so, called by bench.py --calibrate.

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kChains = 8;   // independent accumulators per wave (hides the MFMA latency)

__global__ __launch_bounds__(256) void mfma_loop_bf16(float *out, int iters) {
  const int lane = threadIdx.x & 63;
  bf16x8 a, b;
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(0.001f * (lane + i));
    b[i] = (__bf16)(0.002f * (lane - i));
  }
  floatx4 acc[kChains];
  for (int c = 0; c < kChains; ++c) acc[c] = floatx4{0.f, 0.f, 0.f, 0.f};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < kChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.f;
  for (int c = 0; c < kChains; ++c) s += acc[c][0] + acc[c][1] + acc[c][2] + acc[c][3];
  out[(int64_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

__global__ __launch_bounds__(256) void mfma_loop_f32(float *out, int iters) {
  const int lane = threadIdx.x & 63;
  const float a = 0.001f * lane, b = 0.002f * (64 - lane);
  floatx4 acc[kChains];
  for (int c = 0; c < kChains; ++c) acc[c] = floatx4{0.f, 0.f, 0.f, 0.f};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < kChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.f;
  for (int c = 0; c < kChains; ++c) s += acc[c][0] + acc[c][1] + acc[c][2] + acc[c][3];
  out[(int64_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

__global__ __launch_bounds__(256) void mfma_loop_bf16_32(float *out, int iters) {
  const int lane = threadIdx.x & 63;
  bf16x8 a, b;
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(0.001f * (lane + i));
    b[i] = (__bf16)(0.002f * (lane - i));
  }
  floatx16 acc[kChains];
  for (int c = 0; c < kChains; ++c)
    for (int e = 0; e < 16; ++e) acc[c][e] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < kChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.f;
  for (int c = 0; c < kChains; ++c)
    for (int e = 0; e < 16; ++e) s += acc[c][e];
  out[(int64_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

__global__ __launch_bounds__(256) void mfma_loop_f32_32(float *out, int iters) {
  const int lane = threadIdx.x & 63;
  const float a = 0.001f * lane, b = 0.002f * (64 - lane);
  floatx16 acc[kChains];
  for (int c = 0; c < kChains; ++c)
    for (int e = 0; e < 16; ++e) acc[c][e] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < kChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.f;
  for (int c = 0; c < kChains; ++c)
    for (int e = 0; e < 16; ++e) s += acc[c][e];
  out[(int64_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

// Streaming read: every float4 of src once per launch (grid-stride, two
// loads in flight per lane), summed so the loads are not dropped; one float
// written per lane.  nt: non-temporal loads.
template <bool NT>
__global__ __launch_bounds__(256) void read_stream(const floatx4 *__restrict__ src, int64_t n4, float *out) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  floatx4 a = {0.f, 0.f, 0.f, 0.f}, b = {0.f, 0.f, 0.f, 0.f};
  for (; i + stride < n4; i += 2 * stride) {
    const floatx4 x = NT ? __builtin_nontemporal_load(src + i) : src[i];
    const floatx4 y = NT ? __builtin_nontemporal_load(src + i + stride) : src[i + stride];
    a += x;
    b += y;
  }
  if (i < n4) a += src[i];
  out[(int64_t)blockIdx.x * 256 + threadIdx.x] = a[0] + a[1] + a[2] + a[3] + b[0] + b[1] + b[2] + b[3];
}

}  // namespace

extern "C" {

// Reads `bytes` (a multiple of 16) at src with `blocks` workgroups of 256
// threads (kind 0: cached loads, 1: non-temporal).  out: device float32
// [blocks * 256].  Returns the HIP status of the launch.
int gift_calib_read(void *stream, int kind, const void *src, int64_t bytes, float *out, int blocks) {
  const floatx4 *p = static_cast<const floatx4 *>(src);
  if (kind == 0)
    hipLaunchKernelGGL(read_stream<false>, dim3(blocks), dim3(256), 0, static_cast<hipStream_t>(stream), p, bytes / 16,
                       out);
  else
    hipLaunchKernelGGL(read_stream<true>, dim3(blocks), dim3(256), 0, static_cast<hipStream_t>(stream), p, bytes / 16,
                       out);
  return (int)hipGetLastError();
}

// Launches `blocks` workgroups of 256 threads, each wave running `iters`
// rounds of kChains matrix-core instructions (kind 0: bf16 16x16x32, 16384
// flops each; 1: float32 16x16x4, 2048 flops; 2: bf16 32x32x16, 32768
// flops; 3: float32 32x32x2, 4096 flops).  out: device float32
// [blocks * 256], written once per lane.  Returns the HIP status of the
// launch (invalid kind: hipErrorInvalidValue, nothing launched); flops =
// blocks * 4 * iters * kChains * flops per instruction.
int gift_calib_mfma(void *stream, int kind, float *out, int blocks, int iters) {
  const hipStream_t s = static_cast<hipStream_t>(stream);
  switch (kind) {
    case 0: hipLaunchKernelGGL(mfma_loop_bf16, dim3(blocks), dim3(256), 0, s, out, iters); break;
    case 1: hipLaunchKernelGGL(mfma_loop_f32, dim3(blocks), dim3(256), 0, s, out, iters); break;
    case 2: hipLaunchKernelGGL(mfma_loop_bf16_32, dim3(blocks), dim3(256), 0, s, out, iters); break;
    case 3: hipLaunchKernelGGL(mfma_loop_f32_32, dim3(blocks), dim3(256), 0, s, out, iters); break;
    default: return (int)hipErrorInvalidValue;
  }
  return (int)hipGetLastError();
}

int gift_calib_chains(void) { return kChains; }

}  // extern "C"
