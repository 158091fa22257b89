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

// --------------------------------------------------------- strided leaves
//
// W lanes per row, W a power of two <= 256, lane j folding elements j, j + W,
// j + 2W, ... in index order (Sec. 3.2.2, GEMV: lanes take every count-th
// element).  A row belongs to G = min(W, 64) lanes of one wave (64 / G rows
// per wave); lane q of the group holds the LPL = W / G leaves q LPL ..
// q LPL + LPL - 1, whose elements at step t are the LPL consecutive floats
// from t W + q LPL (one vector load when the row allows it), so every load
// instruction of a wave reads whole contiguous runs.  A leaf without an
// element holds -0, the exact identity of binary32 addition: it joins the
// tree without changing a bit, as an elided addition would.  The tree is
// the perfect tree over the W leaves: in leaf order (DOWN false) the
// in-lane levels (the low leaf bits) come first and then the xor butterfly
// with offsets 1, 2, .., G/2; in bit-reversed order (DOWN true) the
// butterfly runs with offsets G/2, .., 1 first, then the in-lane levels
// from the highest leaf bit down.
template <int W, int OP, bool DOWN, bool VEC>
__global__ __launch_bounds__(256) void rowsum_strided(RowsumArgs a) {
  constexpr int G = W < 64 ? W : 64, LPL = W / G, R = 64 / G;
  constexpr int U = LPL == 4 ? 8 : 16;   // steps whose loads are in flight together
  constexpr int sumsq = OP > 0, fma = OP == 1;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane / G, q = lane % G;
  const int64_t row = ((int64_t)blockIdx.x * RS_WAVES + wave) * R + g;
  const bool live = row < a.rows;
  const int64_t cols = a.cols, nfull = cols / W;
  const float* x = a.X + (live ? row : 0) * cols + q * LPL;

  auto load = [&](int64_t t, float* v) {
    const float* p = x + t * W;
    if constexpr (VEC && LPL == 4) {
      const float4 f = *(const float4*)p;
      v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
    } else if constexpr (VEC && LPL == 2) {
      const float2 f = *(const float2*)p;
      v[0] = f.x; v[1] = f.y;
    } else {
#pragma unroll
      for (int u = 0; u < LPL; ++u) v[u] = p[u];
    }
  };
  float s[LPL];
#pragma unroll
  for (int u = 0; u < LPL; ++u) s[u] = -0.0f;
  if (live && nfull > 0) {
    float v0[LPL];
    load(0, v0);
#pragma unroll
    for (int u = 0; u < LPL; ++u) s[u] = sumsq ? v0[u] * v0[u] : v0[u];
    int64_t t = 1;
    for (; t + U <= nfull; t += U) {
      float v[U][LPL];
#pragma unroll
      for (int i = 0; i < U; ++i) load(t + i, v[i]);
#pragma unroll
      for (int i = 0; i < U; ++i)
#pragma unroll
        for (int u = 0; u < LPL; ++u) s[u] = leaf_step(s[u], v[i][u], sumsq, fma);
    }
    for (; t < nfull; ++t) {
      float v[LPL];
      load(t, v);
#pragma unroll
      for (int u = 0; u < LPL; ++u) s[u] = leaf_step(s[u], v[u], sumsq, fma);
    }
  }
  // the short last step: elements nfull W + q LPL + u below cols
  if (live) {
#pragma unroll
    for (int u = 0; u < LPL; ++u) {
      if (nfull * W + q * LPL + u < cols) {
        const float xv = x[nfull * W + u];
        s[u] = nfull ? leaf_step(s[u], xv, sumsq, fma) : (sumsq ? xv * xv : xv);
      }
    }
  }
  float r;
  if constexpr (!DOWN) {
#pragma unroll
    for (int h = 1; h < LPL; h <<= 1)
#pragma unroll
      for (int u = 0; u < LPL; u += 2 * h) s[u] = s[u] + s[u + h];
    r = s[0];
#pragma unroll
    for (int m = 1; m < G; m <<= 1) r = r + __shfl_xor(r, m, 64);
  } else {
#pragma unroll
    for (int m = G / 2; m >= 1; m >>= 1)
#pragma unroll
      for (int u = 0; u < LPL; ++u) s[u] = s[u] + __shfl_xor(s[u], m, 64);
#pragma unroll
    for (int h = LPL / 2; h >= 1; h >>= 1)
#pragma unroll
      for (int u = 0; u < h; ++u) s[u] = s[u] + s[u + h];
    r = s[0];
  }
  if (live && q == 0) a.out[row] = cols ? r : 0.0f;
}

template <int W, bool DOWN, bool VEC>
static void launch_strided_t(const RowsumArgs& a, int op, hipStream_t st) {
  constexpr int R = 64 / (W < 64 ? W : 64);
  const int64_t per_block = (int64_t)RS_WAVES * R;
  const dim3 grid((unsigned)((a.rows + per_block - 1) / per_block)), block(64 * RS_WAVES);
  if (op == 0) hipLaunchKernelGGL((rowsum_strided<W, 0, DOWN, VEC>), grid, block, 0, st, a);
  else if (op == 1) hipLaunchKernelGGL((rowsum_strided<W, 1, DOWN, VEC>), grid, block, 0, st, a);
  else hipLaunchKernelGGL((rowsum_strided<W, 2, DOWN, VEC>), grid, block, 0, st, a);
}

template <int W, bool DOWN>
static void launch_strided_w(const RowsumArgs& a, int op, hipStream_t st) {
  constexpr int LPL = W > 64 ? W / 64 : 1;
  if constexpr (LPL > 1) {
    if ((((uintptr_t)a.X) % (4 * LPL) == 0) && (a.cols % LPL == 0)) {
      launch_strided_t<W, DOWN, true>(a, op, st);
      return;
    }
  }
  launch_strided_t<W, DOWN, false>(a, op, st);
}

template <bool DOWN>
static hipError_t launch_strided(const RowsumArgs& a, int op, hipStream_t st) {
  switch (a.leaf_w) {
    case 1: launch_strided_w<1, DOWN>(a, op, st); break;
    case 2: launch_strided_w<2, DOWN>(a, op, st); break;
    case 4: launch_strided_w<4, DOWN>(a, op, st); break;
    case 8: launch_strided_w<8, DOWN>(a, op, st); break;
    case 16: launch_strided_w<16, DOWN>(a, op, st); break;
    case 32: launch_strided_w<32, DOWN>(a, op, st); break;
    case 64: launch_strided_w<64, DOWN>(a, op, st); break;
    case 128: launch_strided_w<128, DOWN>(a, op, st); break;
    case 256: launch_strided_w<256, DOWN>(a, op, st); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_rowsum(const RowsumArgs& a, hipStream_t st) {
  if (a.strided) {
    const int op = !a.sumsq ? 0 : a.fma ? 1 : 2;
    return a.down ? launch_strided<true>(a, op, st) : launch_strided<false>(a, op, st);
  }
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
