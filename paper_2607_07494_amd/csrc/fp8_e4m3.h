// OCP FP8 E4M3 (E4M3FN) conversion on the GPU, written from the format
// definition: 1 sign bit, 4 exponent bits (bias 7), 3 mantissa bits,
// subnormals at exponent field 0, largest finite 448 = S.1111.110,
// NaN = S.1111.111, no infinities.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gift {

constexpr float kE4M3Max = 448.0f;

// Round-to-nearest-even E4M3 code of a float, saturating at +-448, keeping
// the sign of zero; NaN -> 0x7F.
__device__ __forceinline__ uint32_t e4m3_encode(float y) {
  const uint32_t u = __float_as_uint(y);
  const uint32_t sign = (u >> 24) & 0x80u;
  const uint32_t a = u & 0x7fffffffu;
  if (a > 0x7f800000u) return 0x7fu;                 // NaN
  if (a >= 0x43e00000u) return sign | 0x7eu;         // |y| >= 448 (and inf)
  if (a < 0x3c800000u) {                             // |y| < 2^-6: spacing 2^-9
    // |y| * 2^9 is exact; rint rounds half to even -> 0..8 (8 = min normal)
    const float t = __uint_as_float(a) * 512.0f;
    return sign | (uint32_t)__builtin_rintf(t);
  }
  // normal binade: drop 20 of the 23 mantissa bits with round-half-even on
  // the exponent|mantissa field (a carry moves into the exponent), then
  // rebias the exponent from 127 to 7.  |y| < 448 keeps the result <= 0x7e.
  const uint32_t rounded = (a + 0x7ffffu + ((a >> 20) & 1u)) >> 20;
  return sign | (rounded - (120u << 3));
}

// Exact float value of an E4M3 code (NaN for 0x7F / 0xFF).
__device__ __forceinline__ float e4m3_decode(uint32_t c) {
  const uint32_t sign = (c & 0x80u) << 24;
  const uint32_t e = (c >> 3) & 0xfu;
  const uint32_t mant = c & 0x7u;
  float v;
  if (e == 0) {
    v = (float)mant * 0.001953125f;                  // mant * 2^-9, exact
  } else {
    v = __uint_as_float(((e + 120u) << 23) | (mant << 20));
  }
  v = __uint_as_float(__float_as_uint(v) | sign);
  return (e == 0xfu && mant == 0x7u) ? __uint_as_float(0x7fc00000u) : v;
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

}  // namespace gift
