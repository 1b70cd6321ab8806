// OCP FP8 E4M3 (E4M3FN) conversion on the GPU: 1 sign bit, 4 exponent bits
// (bias 7), 3 mantissa bits, subnormals at exponent field 0, largest finite
// 448 = S.1111.110, NaN = S.1111.111, no infinities.
//
// gfx950's conversions between float32 and FP8 use the OCP E4M3 format:
// v_cvt_pk_fp8_f32 rounds to nearest even and v_cvt_pk_f32_fp8 is exact.
// The codec's quantizer is "round to nearest even, saturating at +-448,
// keeping the sign of zero, NaN -> 0x7F": the hardware conversion of the value
// clamped to [-448, 448] (clamping keeps -0.0 and maps +-inf to +-448), with
// NaN inputs set to 0x7F afterwards (the clamp would have turned them into
// -448).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gift {

constexpr float kE4M3Max = 448.0f;

__device__ __forceinline__ float e4m3_clamp(float y) { return fminf(fmaxf(y, -kE4M3Max), kE4M3Max); }

// Codes of four floats packed little-endian (value e in byte e).
__device__ __forceinline__ uint32_t e4m3_encode4(float y0, float y1, float y2, float y3) {
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(e4m3_clamp(y0), e4m3_clamp(y1), 0, false);
  w = __builtin_amdgcn_cvt_pk_fp8_f32(e4m3_clamp(y2), e4m3_clamp(y3), w, true);
  uint32_t u = (uint32_t)w;
  if (y0 != y0) u = (u & 0xffffff00u) | 0x0000007fu;
  if (y1 != y1) u = (u & 0xffff00ffu) | 0x00007f00u;
  if (y2 != y2) u = (u & 0xff00ffffu) | 0x007f0000u;
  if (y3 != y3) u = (u & 0x00ffffffu) | 0x7f000000u;
  return u;
}

// Round-to-nearest-even E4M3 code of one float (saturating, sign of zero
// kept, NaN -> 0x7F).
__device__ __forceinline__ uint32_t e4m3_encode(float y) {
  const uint32_t u = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(e4m3_clamp(y), 0.0f, 0, false) & 0xffu;
  return y != y ? 0x7fu : u;
}

// Exact float values of the four codes packed in a word (NaN for 0x7F / 0xFF).
__device__ __forceinline__ void e4m3_decode4(uint32_t w, float v[4]) {
  const auto lo = __builtin_amdgcn_cvt_pk_f32_fp8((int)w, false);
  const auto hi = __builtin_amdgcn_cvt_pk_f32_fp8((int)w, true);
  v[0] = lo[0];
  v[1] = lo[1];
  v[2] = hi[0];
  v[3] = hi[1];
}

// Exact float value of one E4M3 code.
__device__ __forceinline__ float e4m3_decode(uint32_t c) {
  return __builtin_amdgcn_cvt_pk_f32_fp8((int)(c & 0xffu), false)[0];
}

// Stored (dequantization) scale s = fl32(a / 448).
__device__ __forceinline__ float e4m3_scale(float a) { return a / kE4M3Max; }

// Quantization multiplier fl32(448 / a); 0 for a == 0, FLT_MAX on overflow.
__device__ __forceinline__ float e4m3_multiplier(float a) {
  if (a == 0.0f) return 0.0f;
  float inv = kE4M3Max / a;
  if (__float_as_uint(inv) == 0x7f800000u) inv = 3.402823466e38f;
  return inv;
}

// Boundary hits of four codes (Sec. V-C's vulnerability profile): `up`
// counts codes of magnitude 448 (the largest finite value: saturated values
// and the block maximum itself), `lo` counts nonzero inputs whose code is +-0
// (at most half the smallest subnormal after scaling).  NaN inputs count in
// neither.
__device__ __forceinline__ void e4m3_count_hits4(uint32_t packed, float x0, float x1, float x2, float x3,
                                                 uint32_t &up, uint32_t &lo) {
  const float x[4] = {x0, x1, x2, x3};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint32_t mag = (packed >> (8 * e)) & 0x7fu;
    up += mag == 0x7eu;
    lo += (mag == 0u) & (x[e] != 0.0f);
  }
}

// Wave sums of the two counters added to hits[0], hits[1] by lane 0.
__device__ __forceinline__ void e4m3_flush_hits(uint32_t *hits, uint32_t up, uint32_t lo) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    up += (uint32_t)__shfl_xor((int)up, o);
    lo += (uint32_t)__shfl_xor((int)lo, o);
  }
  if ((threadIdx.x & 63) == 0) {
    if (up) atomicAdd(hits, up);
    if (lo) atomicAdd(hits + 1, lo);
  }
}

}  // namespace gift
