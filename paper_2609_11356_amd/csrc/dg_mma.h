// dg_mma.h -- device pieces shared by the GEMM kernels: operand vector
// types, a compile-time loop, the 16x16x32 MFMA wrappers, the per-output
// finish (partial rounding, split-K store or epilogue) and the s_waitcnt
// immediate for vector-memory counts.
#pragma once

#include <type_traits>

#include "dg_device.h"
#include "dg_internal.h"

namespace dg {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short shortx8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Compile-time loop: f(std::integral_constant<int, I>) for I in [B, E), so
// that register arrays indexed by I stay in registers.
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

__device__ __forceinline__ floatx4 mfma16(shortx8 a, shortx8 b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// The fp16 instruction of the same shape (binary16 operands; its chunks
// fold by the same rules, with exponents read from the binary16 fields).
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
__device__ __forceinline__ floatx4 mfma16h(shortx8 a, shortx8 b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                               __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

template <bool F16>
__device__ __forceinline__ floatx4 mfma16t(shortx8 a, shortx8 b, floatx4 c) {
  if constexpr (F16) return mfma16h(a, b, c);
  else return mfma16(a, b, c);
}

// Finish one output: partial rounding, then either the split-K partial store
// or the epilogue (z = y (+) bias_j; optional pre-activation bf16 rounding;
// SiLU; rounding to the output type).
__device__ __forceinline__ void finish(const GemmArgs& a, int s, int64_t i, int64_t j, float y) {
  if (a.partial_bf16) y = round_bf16(y);
  if (a.S > 1) {
    a.ws[((int64_t)s * a.M + i) * a.N + j] = y;
    return;
  }
  float z = y;
  if (a.epilogue != DG_EPI_NONE) z = y + bf16_f32(a.bias[j]);
  if (a.epilogue == DG_EPI_BIAS_SILU) {
    if (a.pre_act) z = round_bf16(z);
    z = silu_f32(z);
  }
  if (a.out_bf16) ((uint16_t*)a.C)[i * a.N + j] = f32_bf16(z);
  else ((float*)a.C)[i * a.N + j] = z;
}

// OCP e4m3 byte(s) widened to bf16 by the part's own conversion (exact:
// every e4m3 value, subnormals and signed zeros included, is a bf16 value;
// NaN stays NaN), the pair in bytes 2h and 2h + 1 of x.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
template <bool HI>
__device__ __forceinline__ uint32_t e4m3x2_bf16x2(uint32_t x) {
  return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)x, 1.0f, HI));
}
__device__ __forceinline__ uint16_t e4m3_bf16(uint8_t b) {
  return (uint16_t)(e4m3x2_bf16x2<false>(b) & 0xffffu);
}

// s_waitcnt immediate waiting for at most n outstanding vector-memory
// operations (gfx9 encoding: vmcnt[3:0] in bits 3:0, vmcnt[5:4] in bits
// 15:14; expcnt 7 and lgkmcnt 15 mean no wait on those counters).
constexpr int vmcnt_only(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

}  // namespace dg
