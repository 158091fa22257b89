// dg_rowsum.hip -- balanced-tree row reduction for gfx950 (paper Sec. 3.1,
// Sec. 5.1).
//
// Order of row r: leaves of leaf_w consecutive elements, each folded in
// index order; the leaves then meet in the balanced tree (neighbours pair
// level by level, an odd last one carried up).  That tree equals the perfect
// tree over the leaves padded on the right with -0 to a power of two (-0 is
// the exact identity of binary32 addition), and the perfect tree over 64
// lanes holding leaves 0..63 in lane order is the count-up xor butterfly
// (offsets 1, 2, 4, .., 32), whose lane steps are DPP and swizzle
// permutations (dg_lanes.h).  So one wave reduces a row in passes of 64
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
#include "dg_lanes.h"

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

__device__ __forceinline__ float butterfly(float v) { return tree_sum_lanes<6>(v); }

// log2 of a power of two up to 64
template <int G>
constexpr int lg2() {
  return G <= 1 ? 0 : 1 + lg2<G / 2>();
}

// One step of a count-down butterfly over an array of per-lane values: each
// value meets its exact partner lane ^ M.
template <int M, int N>
__device__ __forceinline__ void down_step(float* s) {
#pragma unroll
  for (int u = 0; u < N; ++u) s[u] = s[u] + xor_partner<M>(s[u]);
}

// The count-down butterfly's lane steps over groups of G lanes: offsets
// G / 2, ..., 2, 1.
template <int G, int N>
__device__ __forceinline__ void down_lanes(float* s) {
  if constexpr (G >= 64) down_step<32, N>(s);
  if constexpr (G >= 32) down_step<16, N>(s);
  if constexpr (G >= 16) down_step<8, N>(s);
  if constexpr (G >= 8) down_step<4, N>(s);
  if constexpr (G >= 4) down_step<2, N>(s);
  if constexpr (G >= 2) down_step<1, N>(s);
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
  if (live && lane == 0) {
    const float v = have ? r : 0.0f;
    a.out[row] = a.rms == 1 ? rms_inv(v, cols, a.eps) : a.rms == 2 ? 1.0f / v : a.rms == 3 ? v / (float)cols : v;
  }
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
    r = tree_sum_lanes<lg2<G>()>(r);
  } else {
    down_lanes<G, LPL>(s);
#pragma unroll
    for (int h = LPL / 2; h >= 1; h >>= 1)
#pragma unroll
      for (int u = 0; u < h; ++u) s[u] = s[u] + s[u + h];
    r = s[0];
  }
  if (live && q == 0) {
    const float v = cols ? r : 0.0f;
    a.out[row] = a.rms == 1 ? rms_inv(v, cols, a.eps) : a.rms == 2 ? 1.0f / v : a.rms == 3 ? v / (float)cols : v;
  }
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

// ------------------------------------------------------ RMS-norm scaling
//
// out_j = RN_out(y'_j * w_j), y_j = x_j * rinv[row], y'_j = y_j or its bf16
// rounding: elementwise once the row's reciprocal root is known.  One
// workgroup per row; with VEC every thread takes 4 consecutive columns per
// step (16-byte loads of X, 8- or 16-byte stores of Y).
template <bool VEC>
__global__ __launch_bounds__(256) void rmsnorm_scale(NormArgs a) {
  const int64_t row = blockIdx.x, cols = a.cols;
  const float r = a.rinv[row];
  const float* x = a.X + row * cols;
  auto one = [&](float xv, int64_t j) {
    float y = xv * r;
    if (a.pre_round) y = round_bf16(y);
    if (a.w) y = y * bf16_f32(a.w[j]);
    if (a.b) y = y + bf16_f32(a.b[j]);
    return y;
  };
  if (VEC) {
    // U steps of 16-byte loads in flight before any is used
    constexpr int U = 8;
    for (int64_t j0 = 4 * (int64_t)threadIdx.x; j0 < cols; j0 += 1024 * U) {
      float4 xv[U];
#pragma unroll
      for (int i = 0; i < U; ++i) {
        const int64_t j = j0 + 1024 * i;
        xv[i] = j < cols ? *(const float4*)(x + j) : float4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int i = 0; i < U; ++i) {
        const int64_t j = j0 + 1024 * i;
        if (j >= cols) break;
        float y0, y1, y2, y3;
        if (a.w && !a.b && ((uintptr_t)a.w) % 8 == 0) {
          // the four weights in one 8-byte load
          const uint2 q = *(const uint2*)&a.w[j];
          const float xs[4] = {xv[i].x, xv[i].y, xv[i].z, xv[i].w};
          const uint32_t wb[4] = {q.x << 16, q.x & 0xffff0000u, q.y << 16, q.y & 0xffff0000u};
          float ys[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            float y = xs[u] * r;
            if (a.pre_round) y = round_bf16(y);
            ys[u] = y * bits_f32(wb[u]);
          }
          y0 = ys[0]; y1 = ys[1]; y2 = ys[2]; y3 = ys[3];
        } else {
          y0 = one(xv[i].x, j); y1 = one(xv[i].y, j + 1); y2 = one(xv[i].z, j + 2); y3 = one(xv[i].w, j + 3);
        }
        if (a.out_bf16) {
          const uint32_t lo = f32x2_bf16x2(y0, y1);
          const uint32_t hi = f32x2_bf16x2(y2, y3);
          *(uint2*)&((uint16_t*)a.Y)[row * cols + j] = uint2{lo, hi};
        } else {
          *(float4*)&((float*)a.Y)[row * cols + j] = float4{y0, y1, y2, y3};
        }
      }
    }
  } else {
    for (int64_t j = threadIdx.x; j < cols; j += 256) {
      const float y = one(x[j], j);
      if (a.out_bf16) ((uint16_t*)a.Y)[row * cols + j] = f32_bf16(y);
      else ((float*)a.Y)[row * cols + j] = y;
    }
  }
}

// One pass for strided lanes (W = 64, 128, 256) and rows of at most 8192
// elements: one wave per row loads the whole row into registers (lane q
// holds the LPL = W / 64 consecutive floats of every step, at most 128 per
// lane), folds its leaves and meets the other lanes exactly as
// rowsum_strided does, so every lane ends with the row's sum of squares;
// then it scales the values it holds and stores them.  X is read once; the
// weight is staged in LDS once per workgroup.
template <int W, int OP, bool DOWN>
__global__ __launch_bounds__(256) void rmsnorm_strided_fused(RowsumArgs ra, NormArgs a) {
  constexpr int LPL = W / 64, NST = 128 / LPL;
  constexpr int fma = OP == 1;
  __shared__ __attribute__((aligned(16))) uint16_t wl[8192];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t row = (int64_t)blockIdx.x * RS_WAVES + wave;
  const bool live = row < a.rows;
  const int64_t cols = a.cols, nfull = live ? cols / W : 0;
  const float* x = a.X + (live ? row : 0) * cols + lane * LPL;
  if (a.w) {
    if (((uintptr_t)a.w) % 16 == 0 && cols % 8 == 0) {
      for (int64_t j = 8 * (int64_t)threadIdx.x; j < cols; j += 8 * 256) *(uint4*)&wl[j] = *(const uint4*)&a.w[j];
    } else {
      for (int64_t j = threadIdx.x; j < cols; j += 256) wl[j] = a.w[j];
    }
  }
  __syncthreads();
  float v[NST + 1][LPL];
#pragma unroll
  for (int t = 0; t < NST; ++t) {
    if (t < nfull) {
      if constexpr (LPL == 4) {
        const float4 f = *(const float4*)(x + (int64_t)t * W);
        v[t][0] = f.x; v[t][1] = f.y; v[t][2] = f.z; v[t][3] = f.w;
      } else if constexpr (LPL == 2) {
        const float2 f = *(const float2*)(x + (int64_t)t * W);
        v[t][0] = f.x; v[t][1] = f.y;
      } else {
        v[t][0] = x[(int64_t)t * W];
      }
    }
  }
  // the short last step
#pragma unroll
  for (int u = 0; u < LPL; ++u)
    v[NST][u] = (live && nfull * W + lane * LPL + u < cols) ? x[nfull * W + u] : 0.0f;
  float s[LPL];
#pragma unroll
  for (int u = 0; u < LPL; ++u) s[u] = -0.0f;
  if (nfull > 0) {
#pragma unroll
    for (int u = 0; u < LPL; ++u) s[u] = v[0][u] * v[0][u];
  }
#pragma unroll
  for (int t = 1; t < NST; ++t)
    if (t < nfull) {
#pragma unroll
      for (int u = 0; u < LPL; ++u) s[u] = leaf_step(s[u], v[t][u], 1, fma);
    }
#pragma unroll
  for (int u = 0; u < LPL; ++u)
    if (live && nfull * W + lane * LPL + u < cols)
      s[u] = nfull ? leaf_step(s[u], v[NST][u], 1, fma) : v[NST][u] * v[NST][u];
  float r;
  if constexpr (!DOWN) {
#pragma unroll
    for (int h = 1; h < LPL; h <<= 1)
#pragma unroll
      for (int u = 0; u < LPL; u += 2 * h) s[u] = s[u] + s[u + h];
    r = s[0];
    r = tree_sum_lanes<6>(r);
  } else {
    down_lanes<64, LPL>(s);
#pragma unroll
    for (int h = LPL / 2; h >= 1; h >>= 1)
#pragma unroll
      for (int u = 0; u < h; ++u) s[u] = s[u] + s[u + h];
    r = s[0];
  }
  if (!live) return;
  const float rinv = rms_inv(r, cols, ra.eps);
  auto one = [&](float xv, int64_t j) {
    float y = xv * rinv;
    if (a.pre_round) y = round_bf16(y);
    if (a.w) y = y * bf16_f32(wl[j]);
    return y;
  };
  auto put = [&](int64_t j, const float* y, int n) {
    if (a.out_bf16) {
      uint16_t* yp = (uint16_t*)a.Y + row * cols + j;
      if (n == 4) {
        *(uint2*)yp = uint2{f32x2_bf16x2(y[0], y[1]),
                            f32x2_bf16x2(y[2], y[3])};
      } else if (n == 2) {
        *(uint32_t*)yp = f32x2_bf16x2(y[0], y[1]);
      } else {
        for (int u = 0; u < n; ++u) yp[u] = f32_bf16(y[u]);
      }
    } else {
      float* yp = (float*)a.Y + row * cols + j;
      if (n == 4) *(float4*)yp = float4{y[0], y[1], y[2], y[3]};
      else if (n == 2) *(float2*)yp = float2{y[0], y[1]};
      else for (int u = 0; u < n; ++u) yp[u] = y[u];
    }
  };
#pragma unroll
  for (int t = 0; t < NST; ++t)
    if (t < nfull) {
      const int64_t j = (int64_t)t * W + lane * LPL;
      float y[LPL];
      if (a.w) {
        // the step's LPL weights in one LDS read
        uint16_t wv[LPL];
        if constexpr (LPL == 4) {
          const uint2 q = *(const uint2*)&wl[j];
          wv[0] = (uint16_t)q.x; wv[1] = (uint16_t)(q.x >> 16); wv[2] = (uint16_t)q.y; wv[3] = (uint16_t)(q.y >> 16);
        } else if constexpr (LPL == 2) {
          const uint32_t q = *(const uint32_t*)&wl[j];
          wv[0] = (uint16_t)q; wv[1] = (uint16_t)(q >> 16);
        } else {
          wv[0] = wl[j];
        }
#pragma unroll
        for (int u = 0; u < LPL; ++u) {
          float yy = v[t][u] * rinv;
          if (a.pre_round) yy = round_bf16(yy);
          y[u] = yy * bf16_f32(wv[u]);
        }
      } else {
#pragma unroll
        for (int u = 0; u < LPL; ++u) y[u] = one(v[t][u], j + u);
      }
      put(j, y, LPL);
    }
#pragma unroll
  for (int u = 0; u < LPL; ++u) {
    const int64_t j = nfull * W + lane * LPL + u;
    if (j < cols) {
      const float y = one(v[NST][u], j);
      put(j, &y, 1);
    }
  }
}

// The fused pass applies when the row fits the registers and every vector
// access is aligned.
bool rmsnorm_fused_ok(const RowsumArgs& r, const NormArgs& a) {
  const int W = r.leaf_w, LPL = W / 64;
  if (!r.strided || (W != 64 && W != 128 && W != 256) || a.cols > 8192 || a.cols % LPL) return false;
  const int ybytes = a.out_bf16 ? 2 : 4;
  return ((uintptr_t)a.X) % (4 * LPL) == 0 && ((uintptr_t)a.Y) % (ybytes * LPL) == 0;
}

template <int W, bool DOWN>
static void launch_fused_w(const RowsumArgs& r, const NormArgs& a, hipStream_t st) {
  const dim3 grid((unsigned)((a.rows + RS_WAVES - 1) / RS_WAVES)), block(64 * RS_WAVES);
  if (r.fma) hipLaunchKernelGGL((rmsnorm_strided_fused<W, 1, DOWN>), grid, block, 0, st, r, a);
  else hipLaunchKernelGGL((rmsnorm_strided_fused<W, 2, DOWN>), grid, block, 0, st, r, a);
}

hipError_t launch_rmsnorm_fused(const RowsumArgs& r, const NormArgs& a, hipStream_t st) {
  if (r.leaf_w == 64) r.down ? launch_fused_w<64, true>(r, a, st) : launch_fused_w<64, false>(r, a, st);
  else if (r.leaf_w == 128) r.down ? launch_fused_w<128, true>(r, a, st) : launch_fused_w<128, false>(r, a, st);
  else if (r.leaf_w == 256) r.down ? launch_fused_w<256, true>(r, a, st) : launch_fused_w<256, false>(r, a, st);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

// ------------------------------------------------- layer normalisation

// The lanes' partial results meet in the descriptor's tree (W lanes, leaf
// q LPL + u in lane q, slot u): leaf order = in-lane levels then the xor
// butterfly counting up; bit-reversed order = the butterfly counting down
// then the in-lane levels from the highest leaf bit.  Every lane ends with
// the result.
template <int LPL, bool DOWN>
__device__ __forceinline__ float lanes_meet(float (&s)[LPL]) {
  if constexpr (!DOWN) {
#pragma unroll
    for (int h = 1; h < LPL; h <<= 1)
#pragma unroll
      for (int u = 0; u < LPL; u += 2 * h) s[u] = s[u] + s[u + h];
    float r = s[0];
    return tree_sum_lanes<6>(r);
  } else {
    down_lanes<64, LPL>(s);
#pragma unroll
    for (int h = LPL / 2; h >= 1; h >>= 1)
#pragma unroll
      for (int u = 0; u < h; ++u) s[u] = s[u] + s[u + h];
    return s[0];
  }
}

// One pass for strided lanes (W = 64, 128, 256), rows of at most 8192, the
// row in registers as in rmsnorm_strided_fused: the sum (the descriptor's
// leaf folds and tree) gives the mean, the values are centred in place,
// their sum of squares (same order, the fma rule OP) gives the reciprocal
// root, then y = d * rinv, the optional bf16 rounding, weight and bias
// (staged in LDS once per workgroup).
template <int W, int OP, bool DOWN>
__global__ __launch_bounds__(256) void layernorm_strided_fused(RowsumArgs ra, NormArgs a) {
  constexpr int LPL = W / 64, NST = 128 / LPL;
  constexpr int fma = OP == 1;
  __shared__ __attribute__((aligned(16))) uint16_t wl[8192];
  __shared__ __attribute__((aligned(16))) uint16_t bl[8192];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t row = (int64_t)blockIdx.x * RS_WAVES + wave;
  const bool live = row < a.rows;
  const int64_t cols = a.cols, nfull = live ? cols / W : 0;
  const float* x = a.X + (live ? row : 0) * cols + lane * LPL;
  auto stage = [&](const uint16_t* g, uint16_t* l) {
    if (((uintptr_t)g) % 16 == 0 && cols % 8 == 0) {
      for (int64_t j = 8 * (int64_t)threadIdx.x; j < cols; j += 8 * 256) *(uint4*)&l[j] = *(const uint4*)&g[j];
    } else {
      for (int64_t j = threadIdx.x; j < cols; j += 256) l[j] = g[j];
    }
  };
  if (a.w) stage(a.w, wl);
  if (a.b) stage(a.b, bl);
  __syncthreads();
  float v[NST + 1][LPL];
#pragma unroll
  for (int t = 0; t < NST; ++t) {
    if (t < nfull) {
      if constexpr (LPL == 4) {
        const float4 f = *(const float4*)(x + (int64_t)t * W);
        v[t][0] = f.x; v[t][1] = f.y; v[t][2] = f.z; v[t][3] = f.w;
      } else if constexpr (LPL == 2) {
        const float2 f = *(const float2*)(x + (int64_t)t * W);
        v[t][0] = f.x; v[t][1] = f.y;
      } else {
        v[t][0] = x[(int64_t)t * W];
      }
    }
  }
  bool has[LPL];
#pragma unroll
  for (int u = 0; u < LPL; ++u) {
    has[u] = live && nfull * W + lane * LPL + u < cols;
    v[NST][u] = has[u] ? x[nfull * W + u] : 0.0f;
  }
  // the mean
  float s[LPL];
#pragma unroll
  for (int u = 0; u < LPL; ++u) s[u] = nfull ? v[0][u] : -0.0f;
#pragma unroll
  for (int t = 1; t < NST; ++t)
    if (t < nfull)
#pragma unroll
      for (int u = 0; u < LPL; ++u) s[u] = s[u] + v[t][u];
#pragma unroll
  for (int u = 0; u < LPL; ++u)
    if (has[u]) s[u] = nfull ? s[u] + v[NST][u] : v[NST][u];
  const float mean = lanes_meet<LPL, DOWN>(s) / (float)cols;
  // centre in place; the sum of squares of the centred values
#pragma unroll
  for (int t = 0; t < NST; ++t)
    if (t < nfull)
#pragma unroll
      for (int u = 0; u < LPL; ++u) v[t][u] = v[t][u] - mean;
#pragma unroll
  for (int u = 0; u < LPL; ++u)
    if (has[u]) v[NST][u] = v[NST][u] - mean;
#pragma unroll
  for (int u = 0; u < LPL; ++u) s[u] = nfull ? v[0][u] * v[0][u] : -0.0f;
#pragma unroll
  for (int t = 1; t < NST; ++t)
    if (t < nfull)
#pragma unroll
      for (int u = 0; u < LPL; ++u) s[u] = leaf_step(s[u], v[t][u], 1, fma);
#pragma unroll
  for (int u = 0; u < LPL; ++u)
    if (has[u]) s[u] = nfull ? leaf_step(s[u], v[NST][u], 1, fma) : v[NST][u] * v[NST][u];
  const float rinv = rms_inv(lanes_meet<LPL, DOWN>(s), cols, ra.eps);
  if (!live) return;
  auto one = [&](float d, int64_t j) {
    float y = d * rinv;
    if (a.pre_round) y = round_bf16(y);
    if (a.w) y = y * bf16_f32(wl[j]);
    if (a.b) y = y + bf16_f32(bl[j]);
    return y;
  };
  // the LPL bf16 values of a step in one LDS read
  auto chunk = [&](const uint16_t* l, int64_t j, float* out) {
    if constexpr (LPL == 4) {
      const uint2 q = *(const uint2*)&l[j];
      out[0] = bits_f32(q.x << 16); out[1] = bits_f32(q.x & 0xffff0000u);
      out[2] = bits_f32(q.y << 16); out[3] = bits_f32(q.y & 0xffff0000u);
    } else if constexpr (LPL == 2) {
      const uint32_t q = *(const uint32_t*)&l[j];
      out[0] = bits_f32(q << 16); out[1] = bits_f32(q & 0xffff0000u);
    } else {
      out[0] = bf16_f32(l[j]);
    }
  };
#pragma unroll
  for (int t = 0; t < NST; ++t)
    if (t < nfull) {
      const int64_t j = (int64_t)t * W + lane * LPL;
      float y[LPL], wv[LPL], bv[LPL];
      if (a.w) chunk(wl, j, wv);
      if (a.b) chunk(bl, j, bv);
#pragma unroll
      for (int u = 0; u < LPL; ++u) {
        float yy = v[t][u] * rinv;
        if (a.pre_round) yy = round_bf16(yy);
        if (a.w) yy = yy * wv[u];
        if (a.b) yy = yy + bv[u];
        y[u] = yy;
      }
      if (a.out_bf16) {
        uint16_t* yp = (uint16_t*)a.Y + row * cols + j;
        if constexpr (LPL == 4)
          *(uint2*)yp = uint2{f32x2_bf16x2(y[0], y[1]),
                              f32x2_bf16x2(y[2], y[3])};
        else if constexpr (LPL == 2)
          *(uint32_t*)yp = f32x2_bf16x2(y[0], y[1]);
        else
          yp[0] = f32_bf16(y[0]);
      } else {
        float* yp = (float*)a.Y + row * cols + j;
        if constexpr (LPL == 4) *(float4*)yp = float4{y[0], y[1], y[2], y[3]};
        else if constexpr (LPL == 2) *(float2*)yp = float2{y[0], y[1]};
        else yp[0] = y[0];
      }
    }
#pragma unroll
  for (int u = 0; u < LPL; ++u)
    if (has[u]) {
      const int64_t j = nfull * W + lane * LPL + u;
      const float y = one(v[NST][u], j);
      if (a.out_bf16) ((uint16_t*)a.Y)[row * cols + j] = f32_bf16(y);
      else ((float*)a.Y)[row * cols + j] = y;
    }
}

template <int W, bool DOWN>
static void launch_ln_w(const RowsumArgs& r, const NormArgs& a, hipStream_t st) {
  const dim3 grid((unsigned)((a.rows + RS_WAVES - 1) / RS_WAVES)), block(64 * RS_WAVES);
  if (r.fma) hipLaunchKernelGGL((layernorm_strided_fused<W, 1, DOWN>), grid, block, 0, st, r, a);
  else hipLaunchKernelGGL((layernorm_strided_fused<W, 2, DOWN>), grid, block, 0, st, r, a);
}

hipError_t launch_layernorm_fused(const RowsumArgs& r, const NormArgs& a, hipStream_t st) {
  if (r.leaf_w == 64) r.down ? launch_ln_w<64, true>(r, a, st) : launch_ln_w<64, false>(r, a, st);
  else if (r.leaf_w == 128) r.down ? launch_ln_w<128, true>(r, a, st) : launch_ln_w<128, false>(r, a, st);
  else if (r.leaf_w == 256) r.down ? launch_ln_w<256, true>(r, a, st) : launch_ln_w<256, false>(r, a, st);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

// Three-pass path, second pass: the centred values d_j = x_j - mean[row]
// as fp32 into a.Y (a.rinv holds the means).
__global__ __launch_bounds__(256) void layernorm_center(NormArgs a) {
  const int64_t row = blockIdx.x, cols = a.cols;
  const float m = a.rinv[row];
  const float* x = a.X + row * cols;
  float* d = (float*)a.Y + row * cols;
  for (int64_t j = threadIdx.x; j < cols; j += 256) d[j] = x[j] - m;
}

hipError_t launch_layernorm_center(const NormArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(layernorm_center, dim3((unsigned)a.rows), dim3(256), 0, st, a);
  return hipGetLastError();
}

// ------------------------------------------------ GEMM column sums

// The balanced tree down each column of a GEMM output equals the perfect
// tree over the rows padded with -0 (the exact identity) to a power of two,
// so aligned runs of 256 rows are exact subtrees: one thread per (column,
// run) folds its run as a perfect tree (compile-time shape, loads of 16 rows
// in flight), and the run roots meet in the balanced tree (a binary-counter
// stack flushed low to high).  Threads of a wave take consecutive columns,
// so every row load is contiguous across the wave.
constexpr int CS_RUN = 256;

template <bool BF16>
__device__ __forceinline__ float cs_load(const ColsumArgs& a, int64_t i, int64_t j) {
  if constexpr (BF16) return bf16_f32(((const uint16_t*)a.C)[i * a.N + j]);
  else return ((const float*)a.C)[i * a.N + j];
}

template <bool BF16>
__global__ __launch_bounds__(256) void colsum_runs(ColsumArgs a) {
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x, c = blockIdx.y;
  if (j >= a.N) return;
  const int64_t i0 = c * CS_RUN;
  float st[9];            // st[l]: the pending root of 2^l rows
  constexpr int B = 16;   // rows whose loads are in flight together
#pragma unroll
  for (int b = 0; b < CS_RUN / B; ++b) {
    float v[B];
#pragma unroll
    for (int k = 0; k < B; ++k) {
      const int64_t i = i0 + b * B + k;
      v[k] = i < a.M ? cs_load<BF16>(a, i, j) : -0.0f;
    }
    // the perfect tree of the 16 rows, then merged into the run's counter
#pragma unroll
    for (int w = 1; w < B; w <<= 1)
#pragma unroll
      for (int k = 0; k < B; k += 2 * w) v[k] = v[k] + v[k + w];
    float x = v[0];
    int l = 4;                       // 16 = 2^4 rows
#pragma unroll
    for (int bb = b; bb & 1; bb >>= 1) x = st[l++] + x;
    st[l] = x;
  }
  const float root = st[8];
  if (gridDim.y == 1) a.colsum[j] = root;
  else a.part[c * a.N + j] = root;
}

__global__ __launch_bounds__(256) void colsum_merge(ColsumArgs a, int64_t nrun) {
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (j >= a.N) return;
  float st[40];
  uint64_t count = 0;
  for (int64_t c = 0; c < nrun; ++c) {
    float v = a.part[c * a.N + j];
    int l = 0;
    for (uint64_t k = count; k & 1; k >>= 1) v = st[l++] + v;
    st[l] = v;
    ++count;
  }
  float r = 0.0f;
  bool have = false;
  for (int l = 0; l < 40; ++l)
    if ((count >> l) & 1) {
      r = have ? st[l] + r : st[l];
      have = true;
    }
  a.colsum[j] = r;
}

// no rows: every column sums to +0
__global__ __launch_bounds__(256) void colsum_zero(ColsumArgs a) {
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (j < a.N) a.colsum[j] = 0.0f;
}

hipError_t launch_colsum_merge(const ColsumArgs& a, hipStream_t st) {
  const int64_t nrun = (a.M + CS_RUN - 1) / CS_RUN;
  hipLaunchKernelGGL(colsum_merge, dim3((unsigned)((a.N + 255) / 256)), dim3(256), 0, st, a, nrun);
  return hipGetLastError();
}

hipError_t launch_colsum(const ColsumArgs& a, hipStream_t st) {
  if (a.M == 0) {
    hipLaunchKernelGGL(colsum_zero, dim3((unsigned)((a.N + 255) / 256)), dim3(256), 0, st, a);
    return hipGetLastError();
  }
  const int64_t nrun = (a.M + CS_RUN - 1) / CS_RUN;
  const dim3 grid((unsigned)((a.N + 255) / 256), (unsigned)nrun);
  if (a.out_bf16) hipLaunchKernelGGL(colsum_runs<true>, grid, dim3(256), 0, st, a);
  else hipLaunchKernelGGL(colsum_runs<false>, grid, dim3(256), 0, st, a);
  if (nrun > 1) hipLaunchKernelGGL(colsum_merge, dim3((unsigned)((a.N + 255) / 256)), dim3(256), 0, st, a, nrun);
  return hipGetLastError();
}

// ------------------------------------------------------------- softmax

// Maximum with NaN propagation (a NaN operand wins).  Only the sign of a
// zero maximum can depend on the order, and x - (+0) = x - (-0) for every
// x except a zero, whose exp is 1 either way.
__device__ __forceinline__ float max_nan(float a, float b) {
  return (a != a) ? a : (b != b) ? b : (b > a ? b : a);
}

// One pass for strided lanes (W = 64, 128, 256), rows of at most 8192: the
// row in registers as in rmsnorm_strided_fused; the maximum by a butterfly
// (exact), the exponentials in place, their sum folded and met exactly as
// rowsum_strided does (SUM), one reciprocal, one product per element.
template <int W, bool DOWN>
__global__ __launch_bounds__(256) void softmax_strided_fused(RowsumArgs ra, NormArgs a) {
  constexpr int LPL = W / 64, NST = 128 / LPL;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t row = (int64_t)blockIdx.x * RS_WAVES + wave;
  if (row >= a.rows) return;   // whole waves: every shuffle stays inside a live wave
  const int64_t cols = a.cols, nfull = cols / W;
  const float* x = a.X + row * cols + lane * LPL;
  float v[NST + 1][LPL];
#pragma unroll
  for (int t = 0; t < NST; ++t) {
    if (t < nfull) {
      if constexpr (LPL == 4) {
        const float4 f = *(const float4*)(x + (int64_t)t * W);
        v[t][0] = f.x; v[t][1] = f.y; v[t][2] = f.z; v[t][3] = f.w;
      } else if constexpr (LPL == 2) {
        const float2 f = *(const float2*)(x + (int64_t)t * W);
        v[t][0] = f.x; v[t][1] = f.y;
      } else {
        v[t][0] = x[(int64_t)t * W];
      }
    }
  }
  bool has[LPL];   // the short last step's elements present in this lane
#pragma unroll
  for (int u = 0; u < LPL; ++u) {
    has[u] = nfull * W + lane * LPL + u < cols;
    v[NST][u] = has[u] ? x[nfull * W + u] : 0.0f;
  }
  float m = -__builtin_inff();
#pragma unroll
  for (int t = 0; t < NST; ++t)
    if (t < nfull)
#pragma unroll
      for (int u = 0; u < LPL; ++u) m = max_nan(m, v[t][u]);
#pragma unroll
  for (int u = 0; u < LPL; ++u)
    if (has[u]) m = max_nan(m, v[NST][u]);
  m = max_nan(m, butterfly_partner<0>(m));
  m = max_nan(m, butterfly_partner<1>(m));
  m = max_nan(m, butterfly_partner<2>(m));
  m = max_nan(m, butterfly_partner<3>(m));
  m = max_nan(m, butterfly_partner<4>(m));
  m = max_nan(m, butterfly_partner<5>(m));
#pragma unroll
  for (int t = 0; t < NST; ++t)
    if (t < nfull)
#pragma unroll
      for (int u = 0; u < LPL; ++u) v[t][u] = exp_f32(v[t][u] - m);
#pragma unroll
  for (int u = 0; u < LPL; ++u)
    if (has[u]) v[NST][u] = exp_f32(v[NST][u] - m);
  float s[LPL];
#pragma unroll
  for (int u = 0; u < LPL; ++u) s[u] = nfull ? v[0][u] : -0.0f;
#pragma unroll
  for (int t = 1; t < NST; ++t)
    if (t < nfull)
#pragma unroll
      for (int u = 0; u < LPL; ++u) s[u] = s[u] + v[t][u];
#pragma unroll
  for (int u = 0; u < LPL; ++u)
    if (has[u]) s[u] = nfull ? s[u] + v[NST][u] : v[NST][u];
  float r;
  if constexpr (!DOWN) {
#pragma unroll
    for (int h = 1; h < LPL; h <<= 1)
#pragma unroll
      for (int u = 0; u < LPL; u += 2 * h) s[u] = s[u] + s[u + h];
    r = s[0];
    r = tree_sum_lanes<6>(r);
  } else {
    down_lanes<64, LPL>(s);
#pragma unroll
    for (int h = LPL / 2; h >= 1; h >>= 1)
#pragma unroll
      for (int u = 0; u < h; ++u) s[u] = s[u] + s[u + h];
    r = s[0];
  }
  const float rinv = 1.0f / r;
#pragma unroll
  for (int t = 0; t < NST; ++t)
    if (t < nfull) {
      const int64_t j = (int64_t)t * W + lane * LPL;
      float y[LPL];
#pragma unroll
      for (int u = 0; u < LPL; ++u) y[u] = v[t][u] * rinv;
      if (a.out_bf16) {
        uint16_t* yp = (uint16_t*)a.Y + row * cols + j;
        if constexpr (LPL == 4)
          *(uint2*)yp = uint2{f32x2_bf16x2(y[0], y[1]),
                              f32x2_bf16x2(y[2], y[3])};
        else if constexpr (LPL == 2)
          *(uint32_t*)yp = f32x2_bf16x2(y[0], y[1]);
        else
          yp[0] = f32_bf16(y[0]);
      } else {
        float* yp = (float*)a.Y + row * cols + j;
        if constexpr (LPL == 4) *(float4*)yp = float4{y[0], y[1], y[2], y[3]};
        else if constexpr (LPL == 2) *(float2*)yp = float2{y[0], y[1]};
        else yp[0] = y[0];
      }
    }
#pragma unroll
  for (int u = 0; u < LPL; ++u)
    if (has[u]) {
      const int64_t j = nfull * W + lane * LPL + u;
      const float y = v[NST][u] * rinv;
      if (a.out_bf16) ((uint16_t*)a.Y)[row * cols + j] = f32_bf16(y);
      else ((float*)a.Y)[row * cols + j] = y;
    }
}

bool softmax_fused_ok(const RowsumArgs& r, const NormArgs& a) { return rmsnorm_fused_ok(r, a); }

template <int W, bool DOWN>
static void launch_smx_w(const RowsumArgs& r, const NormArgs& a, hipStream_t st) {
  const dim3 grid((unsigned)((a.rows + RS_WAVES - 1) / RS_WAVES)), block(64 * RS_WAVES);
  hipLaunchKernelGGL((softmax_strided_fused<W, DOWN>), grid, block, 0, st, r, a);
}

hipError_t launch_softmax_fused(const RowsumArgs& r, const NormArgs& a, hipStream_t st) {
  if (r.leaf_w == 64) r.down ? launch_smx_w<64, true>(r, a, st) : launch_smx_w<64, false>(r, a, st);
  else if (r.leaf_w == 128) r.down ? launch_smx_w<128, true>(r, a, st) : launch_smx_w<128, false>(r, a, st);
  else if (r.leaf_w == 256) r.down ? launch_smx_w<256, true>(r, a, st) : launch_smx_w<256, false>(r, a, st);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

// Three-pass path, first pass: one workgroup per row finds the maximum
// (order free) and writes e_j = exp(x_j - m) as fp32 to a.Y.
__global__ __launch_bounds__(256) void softmax_exp(NormArgs a) {
  __shared__ float wm[4];
  const int64_t row = blockIdx.x, cols = a.cols;
  const float* x = a.X + row * cols;
  float m = -__builtin_inff();
  for (int64_t j = threadIdx.x; j < cols; j += 256) m = max_nan(m, x[j]);
  m = max_nan(m, butterfly_partner<0>(m));
  m = max_nan(m, butterfly_partner<1>(m));
  m = max_nan(m, butterfly_partner<2>(m));
  m = max_nan(m, butterfly_partner<3>(m));
  m = max_nan(m, butterfly_partner<4>(m));
  m = max_nan(m, butterfly_partner<5>(m));
  if ((threadIdx.x & 63) == 0) wm[threadIdx.x >> 6] = m;
  __syncthreads();
  m = max_nan(max_nan(wm[0], wm[1]), max_nan(wm[2], wm[3]));
  float* e = (float*)a.Y + row * cols;
  for (int64_t j = threadIdx.x; j < cols; j += 256) e[j] = exp_f32(x[j] - m);
}

hipError_t launch_softmax_exp(const NormArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(softmax_exp, dim3((unsigned)a.rows), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_rmsnorm_scale(const NormArgs& a, hipStream_t st) {
  const bool vec = a.cols % 4 == 0 && ((uintptr_t)a.X) % 16 == 0 &&
                   ((uintptr_t)a.Y) % (a.out_bf16 ? 8 : 16) == 0;
  const dim3 grid((unsigned)a.rows), block(256);
  if (vec) hipLaunchKernelGGL((rmsnorm_scale<true>), grid, block, 0, st, a);
  else hipLaunchKernelGGL((rmsnorm_scale<false>), grid, block, 0, st, a);
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
