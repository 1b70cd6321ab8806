// OCP MX FP4 (E2M1) element arithmetic shared by the MXFP4 kernels.
#pragma once

#include <stdint.h>

namespace gift {

// E2M1 magnitude code of a scaled magnitude a: the nearest of 0, 0.5, 1,
// 1.5, 2, 3, 4, 6 with ties to the even code, larger values saturating
__device__ __forceinline__ uint32_t e2m1_mag(float a) {
  return a <= 0.25f ? 0u : a < 0.75f ? 1u : a <= 1.25f ? 2u : a < 1.75f ? 3u
       : a <= 2.5f ? 4u : a < 3.5f ? 5u : a <= 5.0f ? 6u : 7u;
}

// value of an E2M1 magnitude code
__device__ __forceinline__ float e2m1_val(uint32_t mag) {
  return mag < 2u ? 0.5f * (float)mag : (mag < 4u ? 1.0f + 0.5f * (float)(mag - 2u)
                                                  : (mag < 6u ? 2.0f + (float)(mag - 4u) : (mag == 6u ? 4.0f : 6.0f)));
}

// floor(log2(a)) of a finite a > 0 from its bits (subnormals included)
__device__ __forceinline__ int mx_floor_log2(float a) {
  const uint32_t b = __float_as_uint(a);
  const int e = (int)(b >> 23);
  if (e > 0) return e - 127;
  return -149 + (31 - __clz((int)(b & 0x7fffffu)));
}

// scale exponent k of a block (amax over the block, bad = a NaN or an
// infinity in it): 2^k with k = floor(log2 amax) - 2, at least -127
__device__ __forceinline__ int mx_scale_exp(float amax, int bad) {
  int k = -127;
  if (!bad && amax > 0.f) {
    k = mx_floor_log2(amax) - 2;
    k = k < -127 ? -127 : k;
  }
  return k;
}

// code (sign bit 3) and exact dequantized value of v in a block with scale
// exponent k (bad block: code 0, value NaN)
__device__ __forceinline__ uint32_t mx_encode(float v, int k, int bad, float &deq) {
  const uint32_t mag = bad ? 0u : e2m1_mag(fabsf(ldexpf(v, -k)));
  const bool neg = signbit(v);
  const float d = ldexpf(e2m1_val(mag), k);
  deq = bad ? __int_as_float(0x7fc00000) : (neg ? -d : d);
  return bad ? 0u : (mag | (neg ? 8u : 0u));
}

}  // namespace gift
