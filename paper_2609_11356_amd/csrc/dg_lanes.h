// dg_lanes.h -- cross-lane steps of the count-up butterfly on gfx950, built
// from DPP lane permutations (the lowering of the count-up tree on AMD that
// the paper's Sec. 5.1 describes: neighbour exchanges within rows of 16
// lanes, then steps across rows).
//
// A butterfly step pairs every lane with one lane of the other half of its
// 2^(k+1)-lane group; after steps k = 0 .. K-1 every lane holds the perfect
// tree over its 2^K-lane group in lane order (the two operands of a node may
// come in either order: addition commutes, so the bits do not depend on it).
// Any permutation that sends each lane into the other half of its group
// gives that tree once the earlier steps have made the values of each half
// equal, so the steps use the cheapest such permutation:
//   step 0 (lanes 2 apart in pairs):   quad_perm [1, 0, 3, 2]   (xor 1)
//   step 1 (pairs of pairs):           quad_perm [2, 3, 0, 1]   (xor 2)
//   step 2 (quads within 8 lanes):     row_half_mirror (lane k <- 7 - k)
//   step 3 (halves of a 16-lane row):  row_mirror      (lane k <- 15 - k)
//   step 4 (rows 0/1, 2/3):            swizzle xor 16 (ds_swizzle, 32-lane groups)
//   step 5 (the two 32-lane halves):   permute xor 32 (ds_bpermute)
// The DPP forms fold into the add or max that uses them (one instruction per
// step).  The same steps serve a maximum, whose order is free anyway.
#pragma once

#include <hip/hip_runtime.h>

namespace dg {

enum : int {
  kDppXor1 = 0xB1,          // quad_perm [1, 0, 3, 2]
  kDppXor2 = 0x4E,          // quad_perm [2, 3, 0, 1]
  kDppHalfMirror = 0x141,   // row_half_mirror
  kDppMirror = 0x140        // row_mirror
};

template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, true));
}

// The partner of step k (k < 6) of the butterfly.
template <int K>
__device__ __forceinline__ float butterfly_partner(float x) {
  if constexpr (K == 0) return dpp_f32<kDppXor1>(x);
  else if constexpr (K == 1) return dpp_f32<kDppXor2>(x);
  else if constexpr (K == 2) return dpp_f32<kDppHalfMirror>(x);
  else if constexpr (K == 3) return dpp_f32<kDppMirror>(x);
  // ds_swizzle bit mode: and_mask 0x1F, or_mask 0, xor_mask 0x10 (lanes 16 apart
  // within each group of 32)
  else if constexpr (K == 4) return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, x), 0x401F));
  else return __shfl_xor(x, 32, 64);
}

// The exact partner lane ^ M (M a power of two below 64), for butterflies
// whose steps meet lanes that still hold different values (the count-down
// order, whose first step pairs lanes 32 apart): xor 1 and 2 by quad_perm,
// xor 8 by row_ror:8 (a rotation by half of a 16-lane row), xor 4 and 16 by
// ds_swizzle's xor mode (within 32-lane groups), xor 32 by ds_bpermute.
template <int M>
__device__ __forceinline__ float xor_partner(float x) {
  if constexpr (M == 1) return dpp_f32<kDppXor1>(x);
  else if constexpr (M == 2) return dpp_f32<kDppXor2>(x);
  else if constexpr (M == 4) return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, x), 0x101F));
  else if constexpr (M == 8) return dpp_f32<0x128>(x);   // row_ror:8
  else if constexpr (M == 16) return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, x), 0x401F));
  else return __shfl_xor(x, 32, 64);
}

// Sum over groups of 2^K consecutive lanes, the count-up tree in lane order;
// every lane of a group ends with its group's root.
template <int K>
__device__ __forceinline__ float tree_sum_lanes(float x) {
  if constexpr (K >= 1) x = x + butterfly_partner<0>(x);
  if constexpr (K >= 2) x = x + butterfly_partner<1>(x);
  if constexpr (K >= 3) x = x + butterfly_partner<2>(x);
  if constexpr (K >= 4) x = x + butterfly_partner<3>(x);
  if constexpr (K >= 5) x = x + butterfly_partner<4>(x);
  if constexpr (K >= 6) x = x + butterfly_partner<5>(x);
  return x;
}

// Maximum over groups of 2^K consecutive lanes (fmax: a NaN operand is ignored).
template <int K>
__device__ __forceinline__ float max_lanes(float x) {
  if constexpr (K >= 1) x = __builtin_fmaxf(x, butterfly_partner<0>(x));
  if constexpr (K >= 2) x = __builtin_fmaxf(x, butterfly_partner<1>(x));
  if constexpr (K >= 3) x = __builtin_fmaxf(x, butterfly_partner<2>(x));
  if constexpr (K >= 4) x = __builtin_fmaxf(x, butterfly_partner<3>(x));
  if constexpr (K >= 5) x = __builtin_fmaxf(x, butterfly_partner<4>(x));
  if constexpr (K >= 6) x = __builtin_fmaxf(x, butterfly_partner<5>(x));
  return x;
}

}  // namespace dg
