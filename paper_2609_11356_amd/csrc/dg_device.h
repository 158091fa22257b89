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
// keeps its sign and upper payload and gets the quiet bit; overflow carries
// into infinity; subnormals round like any other value.  gfx950's conversion
// instruction (v_cvt_pk_bf16_f32, what the __bf16 cast compiles to) does
// exactly this: it was compared with the bit formula
//   NaN ? (u >> 16) | 0x40 : (u + 0x7fff + ((u >> 16) & 1)) >> 16
// on all 2^32 binary32 inputs on the part, with no difference.
__device__ __forceinline__ uint16_t f32_bf16(float x) { return __builtin_bit_cast(uint16_t, (__bf16)x); }

// Two conversions in one instruction: the low half holds lo, the high half hi.
__device__ __forceinline__ uint32_t f32x2_bf16x2(float lo, float hi) {
  typedef float f2 __attribute__((ext_vector_type(2)));
  typedef __bf16 b2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f2{lo, hi}, b2));
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
//
// Here the steps run on x clamped into [-104, 89] (x itself inside), and the
// scaling is one ldexp: p * 2^(n/2) is exact, so both forms are p * 2^n
// rounded once, and at the clamp ends they give the special values by
// themselves (e^-104 < 2^-150 rounds to 0, 2^128 overflows).  Only a NaN is
// selected separately, so the code has no branches.  This form and the one
// above were compared on all 2^32 binary32 inputs on the part (exp and the
// SiLU built on it), with no difference.
__device__ __forceinline__ float exp_f32(float x_in) {
  const float x = __builtin_fminf(__builtin_fmaxf(x_in, -104.0f), 89.0f);
  const float kLog2e = 0x1.715476p+0f;       // RN32(1 / ln 2)
  const float kLn2Hi = 0x1.62e4p-1f;          // ln 2 rounded to 15 bits
  const float kLn2Lo = 0x1.7f7d1cp-20f;       // RN32(ln 2 - kLn2Hi)
  const float n = __builtin_rintf(x * kLog2e);
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
  const float e = __builtin_ldexpf(p, (int)n);
  return x_in != x_in ? x_in + x_in : e;
}

// 2^x in binary32 by a fixed sequence of steps (the base-two exponential of
// the attention recurrence, whose score scale carries log2 e):
//   n  = rint(x),  f = x - n          (exact, |f| <= 1/2)
//   p  = sum_{k=0..7} c_k f^k,  c_k = RN32((ln 2)^k / k!)   (Horner, fma)
//   2^x = p * 2^n                       (one rounding: the scaling is exact
//                                        but for the last step)
// on x clamped into [-151, 128] (x itself inside): at the clamp ends the
// steps give 0 (2^-151 rounds to zero) and +inf by themselves; a NaN is
// selected at the end, so there are no branches.
__device__ __forceinline__ float exp2_f32(float x_in) {
  const float x = __builtin_fminf(__builtin_fmaxf(x_in, -151.0f), 128.0f);
  const float n = __builtin_rintf(x);
  const float f = x - n;
  float p = 0x1.ffcbfcp-17f;                  // (ln 2)^7 / 7!
  p = __builtin_fmaf(p, f, 0x1.430912p-13f);  // (ln 2)^6 / 6!
  p = __builtin_fmaf(p, f, 0x1.5d87fep-10f);  // (ln 2)^5 / 5!
  p = __builtin_fmaf(p, f, 0x1.3b2ab6p-7f);   // (ln 2)^4 / 4!
  p = __builtin_fmaf(p, f, 0x1.c6b08ep-5f);   // (ln 2)^3 / 3!
  p = __builtin_fmaf(p, f, 0x1.ebfbep-3f);    // (ln 2)^2 / 2!
  p = __builtin_fmaf(p, f, 0x1.62e43p-1f);    // ln 2
  p = __builtin_fmaf(p, f, 1.0f);
  const float e = __builtin_ldexpf(p, (int)n);
  return x_in != x_in ? x_in + x_in : e;
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
