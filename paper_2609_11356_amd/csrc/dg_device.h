// dg_device.h -- device-side scalar helpers shared by the library's kernels.
//
// Every function here is ordinary IEEE binary32 arithmetic (round to nearest
// even, fp32 denormals kept) written so that its bits are fixed by its steps:
// the library is compiled with -ffp-contract=off, and every fused
// multiply-add is spelled out.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dg {

__device__ __forceinline__ float bits_f32(uint32_t u) { return __builtin_bit_cast(float, u); }
__device__ __forceinline__ uint32_t f32_bits(float f) { return __builtin_bit_cast(uint32_t, f); }

__device__ __forceinline__ float bf16_f32(uint16_t h) { return bits_f32((uint32_t)h << 16); }

// binary32 -> bfloat16, round to nearest even on the dropped 16 bits.  A NaN
// keeps its sign and gets the quiet bit; overflow carries into infinity.
__device__ __forceinline__ uint16_t f32_bf16(float x) {
  uint32_t u = f32_bits(x);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

__device__ __forceinline__ float round_bf16(float x) { return bf16_f32(f32_bf16(x)); }

// exp(x) in binary32 by a fixed sequence of steps (Cody & Waite reduction,
// Taylor polynomial, exact power-of-two scaling):
//   n  = rint(x * log2 e)
//   r  = x - n*ln2_hi - n*ln2_lo      (ln2_hi has 15 significant bits, so
//                                      n*ln2_hi is exact for |n| <= 150)
//   p  = sum_{k=0..7} r^k / k!        (Horner, one fma per step)
//   e^x = (p * 2^(n/2)) * 2^(n - n/2)  (two normal powers of two: only the
//                                      last multiply can round)
// Below -104 the result is 0, above 89 it is +inf.
__device__ __forceinline__ float exp_f32(float x) {
  if (x != x) return x + x;
  if (x > 89.0f) return __builtin_inff();
  if (x < -104.0f) return 0.0f;
  const float kLog2e = 0x1.715476p+0f;       // RN32(1 / ln 2)
  const float kLn2Hi = 0x1.62e4p-1f;          // ln 2 rounded to 15 bits
  const float kLn2Lo = 0x1.7f7d1cp-20f;       // RN32(ln 2 - kLn2Hi)
  float n = __builtin_rintf(x * kLog2e);
  float r = __builtin_fmaf(-n, kLn2Hi, x);
  r = __builtin_fmaf(-n, kLn2Lo, r);
  float p = 0x1.a01a02p-13f;                  // RN32(1/7!)
  p = __builtin_fmaf(p, r, 0x1.6c16c2p-10f);  // 1/6!
  p = __builtin_fmaf(p, r, 0x1.111112p-7f);   // 1/5!
  p = __builtin_fmaf(p, r, 0x1.555556p-5f);   // 1/4!
  p = __builtin_fmaf(p, r, 0x1.555556p-3f);   // 1/3!
  p = __builtin_fmaf(p, r, 0.5f);
  p = __builtin_fmaf(p, r, 1.0f);
  p = __builtin_fmaf(p, r, 1.0f);
  int ni = (int)n;
  int n1 = ni / 2, n2 = ni - ni / 2;
  float s1 = bits_f32((uint32_t)(n1 + 127) << 23);
  float s2 = bits_f32((uint32_t)(n2 + 127) << 23);
  return (p * s1) * s2;
}

// SiLU z * sigmoid(z) = z / (1 + exp(-z)), correctly rounded division.
__device__ __forceinline__ float silu_f32(float z) {
  float e = exp_f32(-z);
  return z / (1.0f + e);
}

// RMS-norm reciprocal root of a row's sum of squares s over n = cols
// elements: ms = s / n, v = ms + eps, q = sqrt(v), 1 / q, each one correctly
// rounded binary32 operation (the build keeps IEEE division and sqrt).
__device__ __forceinline__ float rms_inv(float s, int64_t cols, float eps) {
  const float ms = s / (float)cols;
  const float v = ms + eps;
  const float q = __builtin_sqrtf(v);
  return 1.0f / q;
}

}  // namespace dg
