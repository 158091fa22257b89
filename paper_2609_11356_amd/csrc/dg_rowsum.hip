// dg_rowsum.hip -- balanced-tree row reduction for gfx950 (paper Sec. 3.1,
// Sec. 5.1).
//
// Order of row r: leaves of leaf_w consecutive elements, each folded in
// index order; the leaves then meet in the balanced tree (neighbours pair
// level by level, an odd last one carried up).  That tree equals the perfect
// tree over the leaves padded on the right with -0 to a power of two (-0 is
// the exact identity of binary32 addition), and the perfect tree over 64
// lanes holding leaves 0..63 in lane order is the count-up xor butterfly
// (offsets 1, 2, 4, .., 32).  So one wave reduces a row in passes of 64
// leaves: every lane folds one leaf, the butterfly gives the pass root, and
// the pass roots are combined by the same tree through a binary-counter
// stack (lane k of the wave holds level k).
//
// Layout (free once the tree is pinned, Sec. 5.2): a pass's 64 leaves are
// read from HBM with coalesced 16-byte loads and written to LDS with a
// one-element skew per leaf (leaf stride leaf_w + 1), so that the lane-wise
// sequential leaf reads are free of bank conflicts.  Leaves wider than 64
// elements are folded straight from global memory.
#include "dg_device.h"
#include "dg_internal.h"

namespace dg {

constexpr int RS_WAVES = 4;            // rows per workgroup (one per wave)
constexpr int RS_LDS = 64 * 65;        // floats per wave: 64 leaves x (64 + 1)

__device__ __forceinline__ float leaf_step(float s, float x, int sumsq, int fma) {
  if (!sumsq) return s + x;
  if (fma) return __builtin_fmaf(x, x, s);
  float q = x * x;
  return s + q;
}

// The waves of a workgroup reduce different rows in disjoint LDS regions, so
// no workgroup barrier is needed: a wave waits for its own LDS operations
// (lgkmcnt(0)) before the next phase touches the same locations.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_s_waitcnt(0xc07f);
  __builtin_amdgcn_wave_barrier();
}

__device__ __forceinline__ float butterfly(float v) {
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) v = v + __shfl_xor(v, m, 64);
  return v;
}

// Staged path (leaf_w <= 64, 16-byte aligned rows): a pass's 64 leaves are
// fetched with all of the pass's 16-byte loads in flight at once (a lane
// holds leaf_w floats of the pass in registers), the next pass's loads are
// issued before the current pass is folded, and LDS is only the transpose.
// LW: the leaf width when fixed at compile time, else 0.  OP: 0 SUM, 1 SUMSQ
// with fused square-add, 2 SUMSQ with a rounded square, -1 read from a.
template <bool VEC, int LW, int OP>
__global__ __launch_bounds__(256) void rowsum_kernel(RowsumArgs a) {
  const int sumsq = OP < 0 ? a.sumsq : OP > 0, fma = OP < 0 ? a.fma : OP == 1;
  __shared__ float lds[RS_WAVES][RS_LDS];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t row = (int64_t)blockIdx.x * RS_WAVES + wave;
  const bool live = row < a.rows;
  const int lw = LW ? LW : a.leaf_w;
  const int64_t cols = a.cols;
  const int64_t L = (cols + lw - 1) / lw;
  const int64_t npass = (L + 63) / 64;
  const float* x = a.X + (live ? row : 0) * cols;
  const bool staged = lw <= 64;
  float* sl = lds[wave];

  float4 cur[16];
  // pass p holds elements [p*64*lw, p*64*lw + nel); lane takes elements
  // 4*lane + 256*i (i < 16) of it
  auto fetch = [&](int64_t p, float4* r) {
    const int64_t base = p * 64 * lw;
    const int nel = (int)((cols - base < 64 * (int64_t)lw) ? cols - base : 64 * (int64_t)lw);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int e = 4 * lane + 256 * i;
      r[i] = (live && e < nel) ? *(const float4*)(x + base + e) : float4{0.f, 0.f, 0.f, 0.f};
    }
  };
  if (VEC && staged && npass > 0) fetch(0, cur);

  float stackv = 0.f;   // lane k: level k of the pass-root stack
  uint32_t count = 0;
  for (int64_t p = 0; p < npass; ++p) {
    const int64_t base = p * 64 * lw;                   // first element of the pass
    const int nel = (int)((cols - base < 64 * (int64_t)lw) ? cols - base : 64 * (int64_t)lw);
    const int64_t leaf = p * 64 + lane;
    float s = -0.0f;                                    // padding leaf
    if (staged) {
      if (VEC) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int e = 4 * lane + 256 * i;
          if (e < nel) {
            const float vv[4] = {cur[i].x, cur[i].y, cur[i].z, cur[i].w};
#pragma unroll
            for (int q = 0; q < 4; ++q) sl[((e + q) / lw) * (lw + 1) + (e + q) % lw] = vv[q];
          }
        }
      } else if (live) {
        for (int el = lane; el < nel; el += 64) sl[(el / lw) * (lw + 1) + el % lw] = x[base + el];
      }
      wave_lds_sync();
      // cur has been written to LDS: reuse it for the next pass's loads,
      // which stay in flight while this pass is folded
      if (VEC && p + 1 < npass) fetch(p + 1, cur);
      if (live && leaf < L) {
        const int n = (int)((cols - leaf * lw < lw) ? cols - leaf * lw : lw);
        const float* lp = sl + lane * (lw + 1);
        float x0 = lp[0];
        s = sumsq ? x0 * x0 : x0;
        for (int i = 1; i < n; ++i) s = leaf_step(s, lp[i], sumsq, fma);
      }
      wave_lds_sync();
    } else if (live && leaf < L) {
      const int64_t n = (cols - leaf * lw < lw) ? cols - leaf * lw : lw;
      const float* lp = x + leaf * lw;
      float x0 = lp[0];
      s = sumsq ? x0 * x0 : x0;
      for (int64_t i = 1; i < n; ++i) s = leaf_step(s, lp[i], sumsq, fma);
    }
    float v = butterfly(s);                             // root of this pass
    // push onto the binary-counter stack (uniform across the wave)
    uint32_t c = count;
    int lvl = 0;
    while (c & 1u) {
      v = __shfl(stackv, lvl, 64) + v;
      c >>= 1;
      ++lvl;
    }
    if (lane == lvl) stackv = v;
    ++count;
  }
  // flush low -> high
  float r = 0.0f;
  bool have = false;
  for (int lvl = 0; lvl < 32; ++lvl) {
    if ((count >> lvl) & 1u) {
      const float sv = __shfl(stackv, lvl, 64);
      r = have ? sv + r : sv;
      have = true;
    }
  }
  if (live && lane == 0) a.out[row] = have ? r : 0.0f;
}

hipError_t launch_rowsum(const RowsumArgs& a, hipStream_t st) {
  const int64_t blocks = (a.rows + RS_WAVES - 1) / RS_WAVES;
  const bool vec = ((((uintptr_t)a.X) & 15) == 0) && (a.cols % 4 == 0);
  const dim3 grid((unsigned)blocks), block(64 * RS_WAVES);
  const int op = !a.sumsq ? 0 : a.fma ? 1 : 2;
  if (vec && a.leaf_w == 64) {
    if (op == 0) hipLaunchKernelGGL((rowsum_kernel<true, 64, 0>), grid, block, 0, st, a);
    else if (op == 1) hipLaunchKernelGGL((rowsum_kernel<true, 64, 1>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((rowsum_kernel<true, 64, 2>), grid, block, 0, st, a);
  } else if (vec) {
    hipLaunchKernelGGL((rowsum_kernel<true, 0, -1>), grid, block, 0, st, a);
  } else {
    hipLaunchKernelGGL((rowsum_kernel<false, 0, -1>), grid, block, 0, st, a);
  }
  return hipGetLastError();
}

}  // namespace dg
