// Peak calibration kernels for the benchmark's roofline (not part of the
// codec): matrix-core loops with no memory traffic, whose rate is the
// achievable dense MFMA throughput of this GPU for the two instruction kinds
// the codec uses (bf16 16x16x32 for the statistics and the split-bf16
// transforms, float32 16x16x4 for the inverse transform).  Built into
// libgift_calib.so, called by bench.py --calibrate.

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
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

}  // namespace

extern "C" {

// Launches `blocks` workgroups of 256 threads, each wave running `iters`
// rounds of kChains matrix-core instructions (kind 0: bf16 16x16x32, 16384
// flops each; kind 1: float32 16x16x4, 2048 flops each).  out: device
// float32 [blocks * 256], written once per lane.  Returns the HIP status of
// the launch; flops = blocks * 4 * iters * kChains * flops per instruction.
int gift_calib_mfma(void *stream, int kind, float *out, int blocks, int iters) {
  if (kind == 0)
    hipLaunchKernelGGL(mfma_loop_bf16, dim3(blocks), dim3(256), 0, static_cast<hipStream_t>(stream), out, iters);
  else
    hipLaunchKernelGGL(mfma_loop_f32, dim3(blocks), dim3(256), 0, static_cast<hipStream_t>(stream), out, iters);
  return (int)hipGetLastError();
}

int gift_calib_chains(void) { return kChains; }

}  // extern "C"
