// Wave-level sums of x[0..63] (one wave of 64 lanes) written several ways,
// for the static order checker: the lane steps of the library (dg_lanes.h)
// and hand-written alternatives.  Compiled to gfx950 assembly only; never
// launched.
#include <hip/hip_runtime.h>

#include "../../paper_2609_11356_amd/csrc/dg_lanes.h"

#define KERNEL extern "C" __global__ void __launch_bounds__(64)

// the count-up tree as the library lowers it (DPP, ds_swizzle, ds_bpermute)
KERNEL up_library(const float* __restrict__ x, float* __restrict__ y) {
  const int l = threadIdx.x;
  y[l] = dg::tree_sum_lanes<6>(x[l]);
}

// the same tree with every step a __shfl_xor
KERNEL up_shfl(const float* __restrict__ x, float* __restrict__ y) {
  const int l = threadIdx.x;
  float v = x[l];
  for (int m = 1; m < 64; m <<= 1) v = v + __shfl_xor(v, m, 64);
  y[l] = v;
}

// four consecutive elements per lane (pairwise in the lane), 16 lanes
KERNEL up_four(const float* __restrict__ x, float* __restrict__ y) {
  const int l = threadIdx.x;
  if (l < 16) {
    const float a = x[4 * l], b = x[4 * l + 1], c = x[4 * l + 2], d = x[4 * l + 3];
    const float v = dg::tree_sum_lanes<4>((a + b) + (c + d));
    if (l == 0) y[0] = v;
  }
}

// two consecutive elements per lane, 32 lanes
KERNEL up_two(const float* __restrict__ x, float* __restrict__ y) {
  const int l = threadIdx.x;
  if (l < 32) {
    const float v = dg::tree_sum_lanes<5>(x[2 * l] + x[2 * l + 1]);
    if (l == 0) y[0] = v;
  }
}

// lanes read the elements in reverse order: every node's operands swap,
// which addition's commutativity allows
KERNEL up_reversed(const float* __restrict__ x, float* __restrict__ y) {
  const int l = threadIdx.x;
  const float v = dg::tree_sum_lanes<6>(x[63 - l]);
  if (l == 0) y[0] = v;
}

// the count-down fold (lanes 32 apart first), the library's xor partners
KERNEL down_library(const float* __restrict__ x, float* __restrict__ y) {
  const int l = threadIdx.x;
  float v = x[l];
  v = v + dg::xor_partner<32>(v);
  v = v + dg::xor_partner<16>(v);
  v = v + dg::xor_partner<8>(v);
  v = v + dg::xor_partner<4>(v);
  v = v + dg::xor_partner<2>(v);
  v = v + dg::xor_partner<1>(v);
  y[l] = v;
}

// the count-down fold with every step a __shfl_xor
KERNEL down_shfl(const float* __restrict__ x, float* __restrict__ y) {
  const int l = threadIdx.x;
  float v = x[l];
  for (int m = 32; m >= 1; m >>= 1) v = v + __shfl_xor(v, m, 64);
  y[l] = v;
}

// a plausible slip: the first two steps swapped (lanes 2 apart, then 1)
KERNEL up_steps_swapped(const float* __restrict__ x, float* __restrict__ y) {
  const int l = threadIdx.x;
  float v = x[l];
  v = v + __shfl_xor(v, 2, 64);
  v = v + __shfl_xor(v, 1, 64);
  for (int m = 4; m < 64; m <<= 1) v = v + __shfl_xor(v, m, 64);
  y[l] = v;
}

// a left fold in one lane
KERNEL chain(const float* __restrict__ x, float* __restrict__ y) {
  if (threadIdx.x == 0) {
    float v = x[0];
#pragma unroll
    for (int i = 1; i < 64; ++i) v = v + x[i];
    y[0] = v;
  }
}

// groups of 16 lanes: four sums, one per group (the row sums of a 16-lane
// row group, as in the attention kernel's block row sum)
KERNEL groups16(const float* __restrict__ x, float* __restrict__ y) {
  const int l = threadIdx.x;
  const float v = dg::tree_sum_lanes<4>(x[l]);
  if ((l & 15) == 0) y[l >> 4] = v;
}

// an instruction the walk does not model (the hardware reciprocal): an
// uninterpreted function of its operand, so each lane's leaf stays distinct
KERNEL rcp_then_up(const float* __restrict__ x, float* __restrict__ y) {
  const int l = threadIdx.x;
  y[l] = dg::tree_sum_lanes<6>(__builtin_amdgcn_rcpf(x[l]));
}

// control flow that depends on the data: the walk refuses it
KERNEL branch_on_data(const float* __restrict__ x, float* __restrict__ y) {
  const int l = threadIdx.x;
  float v = x[l];
  if (v > 0.f) v = dg::tree_sum_lanes<6>(v);
  y[l] = v;
}

// a workgroup's sum of x[0..255]: each wave's tree over its 64 elements, the
// four wave sums through LDS, then a tree over them in wave order
extern "C" __global__ void __launch_bounds__(256) block_256(const float* __restrict__ x, float* __restrict__ y) {
  __shared__ float part[4];
  const int t = threadIdx.x, l = t & 63, w = t >> 6;
  const float v = dg::tree_sum_lanes<6>(x[t]);
  if (l == 0) part[w] = v;
  __syncthreads();
  if (t < 4) {
    const float s = dg::tree_sum_lanes<2>(part[t]);
    if (t == 0) y[0] = s;
  }
}

// the same tree from 128 threads holding two consecutive elements each (the
// cut between in-thread, in-wave and cross-wave levels moves)
extern "C" __global__ void __launch_bounds__(128) block_128x2(const float* __restrict__ x, float* __restrict__ y) {
  __shared__ float part[2];
  const int t = threadIdx.x, l = t & 63, w = t >> 6;
  const float v = dg::tree_sum_lanes<6>(x[2 * t] + x[2 * t + 1]);
  if (l == 0) part[w] = v;
  __syncthreads();
  if (t == 0) y[0] = part[0] + part[1];
}

// the wave sums chained in wave order
extern "C" __global__ void __launch_bounds__(256) block_256_chain(const float* __restrict__ x, float* __restrict__ y) {
  __shared__ float part[4];
  const int t = threadIdx.x, l = t & 63, w = t >> 6;
  const float v = dg::tree_sum_lanes<6>(x[t]);
  if (l == 0) part[w] = v;
  __syncthreads();
  if (t == 0) y[0] = ((part[0] + part[1]) + part[2]) + part[3];
}

// loops over n (bound to a configuration by the caller): lane l folds
// x[l], x[l + 64], x[l + 128], ... in order, then the count-up tree
KERNEL strided_fold(const float* __restrict__ x, float* __restrict__ y, int n) {
  const int l = threadIdx.x;
  float v = x[l];
#pragma nounroll
  for (int k = l + 64; k < n; k += 64) v = v + x[k];
  y[l] = dg::tree_sum_lanes<6>(v);
}

// the same chain unrolled by two (one accumulator): the same tree
KERNEL strided_fold_unroll2(const float* __restrict__ x, float* __restrict__ y, int n) {
  const int l = threadIdx.x;
  float v = x[l];
  int k = l + 64;
#pragma nounroll
  for (; k + 64 < n; k += 128) {
    v = v + x[k];
    v = v + x[k + 64];
  }
  if (k < n) v = v + x[k];
  y[l] = dg::tree_sum_lanes<6>(v);
}

// two accumulators (even and odd steps) joined at the end: re-chunking a
// sequential fold regroups the sum
KERNEL strided_fold_two_acc(const float* __restrict__ x, float* __restrict__ y, int n) {
  const int l = threadIdx.x;
  float v0 = x[l], v1 = x[l + 64];
  int k = l + 128;
#pragma nounroll
  for (; k + 64 < n; k += 128) {
    v0 = v0 + x[k];
    v1 = v1 + x[k + 64];
  }
  y[l] = dg::tree_sum_lanes<6>(v0 + v1);
}
