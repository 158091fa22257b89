// dg_gemm.hip -- GEMM kernels for gfx950 whose reduction order is the
// descriptor's (paper Sec. 3.2.2), independent of tile shape and grid.
//
// Arithmetic of one bf16 MFMA on gfx950 (measured; used here only as the
// unit the order is built from): v_mfma_f32_16x16x32_bf16 folds its 32 k in
// four chunks of 8 consecutive k, lanes 16c..16c+15 carrying chunk c
// (k = 8c..8c+7 of the instruction's K slice), each chunk updating the
// accumulator with one rounding, chunk 0 first.  A chunk whose products are
// all zero leaves the accumulator as it is.  Two consequences shape every
// kernel below:
//   * with the accumulator as C operand (fma = 1) the order is the chain of
//     8-k chunks, cut from each tile start; any instruction sequence that
//     walks those chunks in increasing k gives the same bits, so the K step
//     per instruction, the LDS staging and the tile shape are free;
//   * zero padding (k past a tile or part end, rows past M, columns past N)
//     never changes an accumulator, so operands can be zero-filled freely.
//
// Kernels:
//   gemm_generic     any descriptor: one wave per 16x16 output block and
//                    part; element loads; per-tile combine (carry, chain,
//                    balanced tree via a binary-counter stack in LDS).
//   gemm_tiled<...>  carried accumulator (tile_combine CARRY, fma = 1) with
//                    8-aligned chunks: BMxBN block per workgroup, 4 waves,
//                    global -> registers -> LDS double buffer (B transposed
//                    in registers on the way), 16x16x32 MFMA.
//   splitk_combine   S fp32 partials -> chain or balanced tree at the merge
//                    precision -> epilogue (no atomics: the second kernel on
//                    the same stream).
#include "dg_device.h"
#include "dg_internal.h"

namespace dg {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short shortx8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ floatx4 mfma16(shortx8 a, shortx8 b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
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

// ------------------------------------------------------------- generic

__global__ __launch_bounds__(64) void gemm_generic(GemmArgs a) {
  __shared__ floatx4 stk[32][64];  // binary-counter stack for the tile tree
  const int lane = threadIdx.x;
  const int64_t i0 = (int64_t)blockIdx.y * 16, j0 = (int64_t)blockIdx.x * 16;
  const int s = blockIdx.z;
  const int64_t k0 = a.cuts[s], k1 = a.cuts[s + 1];
  const int64_t len = k1 - k0, tk = a.tile_k;
  const int64_t ntiles = (len + tk - 1) / tk;
  int64_t first = tk;
  if (a.tail_first && (len % tk)) first = len % tk;
  const int64_t arow = i0 + (lane & 15), bcol = j0 + (lane & 15);
  const int kb = 8 * (lane >> 4);
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
  const int64_t step = a.fma ? 32 : a.group;  // one instruction per step
  floatx4 acc = zero;
  uint32_t count = 0;
  int64_t ts = k0;
  for (int64_t t = 0; t < ntiles; ++t) {
    int64_t tl = (t == 0) ? (first < len ? first : len) : tk;
    if (ts + tl > k1) tl = k1 - ts;
    const int64_t te = ts + tl;
    floatx4 v = (a.tile_combine == DG_CARRY) ? acc : zero;
    for (int64_t gs = ts; gs < te; gs += step) {
      const int64_t ge = (gs + step < te) ? gs + step : te;
      shortx8 av, bv;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int64_t k = gs + kb + e;
        const bool ok = k < ge;
        av[e] = (ok && arow < a.M) ? (short)a.A[arow * a.K + k] : (short)0;
        bv[e] = (ok && bcol < a.N) ? (short)a.B[k * a.N + bcol] : (short)0;
      }
      if (a.fma) {
        v = mfma16(av, bv, v);
      } else {
        floatx4 w = mfma16(av, bv, zero);
        v = v + w;
      }
    }
    if (a.tile_combine == DG_CARRY) {
      acc = v;
    } else if (a.tile_combine == DG_SEQ) {
      acc = (t == 0) ? v : acc + v;
    } else {
      uint32_t c = count;
      int lvl = 0;
      while (c & 1u) {
        v = stk[lvl][lane] + v;
        c >>= 1;
        ++lvl;
      }
      stk[lvl][lane] = v;
      ++count;
    }
    ts = te;
  }
  if (a.tile_combine == DG_TREE && count) {
    bool have = false;
    for (int lvl = 0; lvl < 32; ++lvl) {
      if ((count >> lvl) & 1u) {
        acc = have ? stk[lvl][lane] + acc : stk[lvl][lane];
        have = true;
      }
    }
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int64_t i = i0 + 4 * (lane >> 4) + r;
    if (i < a.M && bcol < a.N) finish(a, s, i, bcol, acc[r]);
  }
}

// --------------------------------------------------------------- tiled

constexpr int BK = 64;
constexpr int LDS_PITCH = BK + 8;  // bf16 elements per LDS row (16 B pad)

// A 16-byte vector of A row `row` at k..k+7, zero past M or past the part end.
__device__ __forceinline__ uint4 load_a_vec(const GemmArgs& a, int64_t row, int64_t k, int64_t k1) {
  uint4 r = {0u, 0u, 0u, 0u};
  if (row >= a.M || k >= k1) return r;
  const uint16_t* p = a.A + row * a.K + k;
  if (k + 8 <= k1) return *(const uint4*)p;
  uint16_t t[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) t[e] = (k + e < k1) ? p[e] : (uint16_t)0;
  return __builtin_bit_cast(uint4, t);
}

// A 16-byte vector of B row k at columns n..n+7 (N % 8 == 0: all or none).
__device__ __forceinline__ uint4 load_b_vec(const GemmArgs& a, int64_t k, int64_t n, int64_t k1) {
  uint4 r = {0u, 0u, 0u, 0u};
  if (k >= k1 || n >= a.N) return r;
  return *(const uint4*)(a.B + k * a.N + n);
}

template <int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(256) void gemm_tiled(GemmArgs a) {
  static_assert(WM * WN == 4, "four waves");
  constexpr int WTM = BM / WM, WTN = BN / WN;  // rows / cols per wave
  constexpr int TM = WTM / 16, TN = WTN / 16;  // 16x16 MFMA blocks per wave
  static_assert(TM >= 1 && TN >= 1 && WTM % 16 == 0 && WTN % 16 == 0, "wave tile");
  constexpr int AV = BM * (BK / 8);            // 16 B vectors in an A slab
  constexpr int BB = (BK / 4) * (BN / 8);      // 4x8 blocks in a B slab
  constexpr int AV_T = (AV + 255) / 256, BB_T = (BB + 255) / 256;

  __shared__ __attribute__((aligned(16))) uint16_t As[2][BM][LDS_PITCH];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BN][LDS_PITCH];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int64_t i0 = (int64_t)blockIdx.y * BM, j0 = (int64_t)blockIdx.x * BN;
  const int s = blockIdx.z;
  const int64_t k0 = a.cuts[s], k1 = a.cuts[s + 1];
  const int nslab = (int)((k1 - k0 + BK - 1) / BK);

  floatx4 acc[TM][TN];
#pragma unroll
  for (int mi = 0; mi < TM; ++mi)
#pragma unroll
    for (int ni = 0; ni < TN; ++ni) acc[mi][ni] = floatx4{0.f, 0.f, 0.f, 0.f};

  uint4 ra[AV_T];
  uint4 rb[BB_T][4];

  auto gload = [&](int64_t ks) {
#pragma unroll
    for (int t = 0; t < AV_T; ++t) {
      const int v = tid + 256 * t;
      if (AV % 256 == 0 || v < AV) ra[t] = load_a_vec(a, i0 + v / (BK / 8), ks + 8 * (v % (BK / 8)), k1);
    }
#pragma unroll
    for (int t = 0; t < BB_T; ++t) {
      const int b = tid + 256 * t;
      if (BB % 256 == 0 || b < BB) {
        const int kq = b % (BK / 4), nb = b / (BK / 4);
#pragma unroll
        for (int q = 0; q < 4; ++q) rb[t][q] = load_b_vec(a, ks + 4 * kq + q, j0 + 8 * nb, k1);
      }
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int t = 0; t < AV_T; ++t) {
      const int v = tid + 256 * t;
      if (AV % 256 == 0 || v < AV)
        *(uint4*)&As[buf][v / (BK / 8)][8 * (v % (BK / 8))] = ra[t];
    }
#pragma unroll
    for (int t = 0; t < BB_T; ++t) {
      const int b = tid + 256 * t;
      if (BB % 256 == 0 || b < BB) {
        const int kq = b % (BK / 4), nb = b / (BK / 4);
        const uint32_t* r0 = (const uint32_t*)&rb[t][0];
        const uint32_t* r1 = (const uint32_t*)&rb[t][1];
        const uint32_t* r2 = (const uint32_t*)&rb[t][2];
        const uint32_t* r3 = (const uint32_t*)&rb[t][3];
        // column n = 8nb + u holds k = 4kq .. 4kq+3 -> one 8-byte row piece
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int d = u >> 1;
          uint32_t lo, hi;
          if (u & 1) {
            lo = (r0[d] >> 16) | (r1[d] & 0xffff0000u);
            hi = (r2[d] >> 16) | (r3[d] & 0xffff0000u);
          } else {
            lo = (r0[d] & 0xffffu) | (r1[d] << 16);
            hi = (r2[d] & 0xffffu) | (r3[d] << 16);
          }
          *(uint2*)&Bs[buf][8 * nb + u][4 * kq] = uint2{lo, hi};
        }
      }
    }
  };

  if (nslab > 0) {
    gload(k0);
    lstore(0);
  }
  __syncthreads();
  for (int sl = 0; sl < nslab; ++sl) {
    const int buf = sl & 1;
    if (sl + 1 < nslab) gload(k0 + (int64_t)(sl + 1) * BK);
#pragma unroll
    for (int kk = 0; kk < BK; kk += 32) {
      shortx8 af[TM], bfr[TN];
#pragma unroll
      for (int mi = 0; mi < TM; ++mi)
        af[mi] = *(const shortx8*)&As[buf][wm * WTM + 16 * mi + (lane & 15)][kk + 8 * (lane >> 4)];
#pragma unroll
      for (int ni = 0; ni < TN; ++ni)
        bfr[ni] = *(const shortx8*)&Bs[buf][wn * WTN + 16 * ni + (lane & 15)][kk + 8 * (lane >> 4)];
#pragma unroll
      for (int mi = 0; mi < TM; ++mi)
#pragma unroll
        for (int ni = 0; ni < TN; ++ni) acc[mi][ni] = mfma16(af[mi], bfr[ni], acc[mi][ni]);
    }
    if (sl + 1 < nslab) lstore(buf ^ 1);
    __syncthreads();
  }

#pragma unroll
  for (int mi = 0; mi < TM; ++mi)
#pragma unroll
    for (int ni = 0; ni < TN; ++ni) {
      const int64_t j = j0 + wn * WTN + 16 * ni + (lane & 15);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t i = i0 + wm * WTM + 16 * mi + 4 * (lane >> 4) + r;
        if (i < a.M && j < a.N) finish(a, s, i, j, acc[mi][ni][r]);
      }
    }
}

// ------------------------------------------------------- split-K merge

__global__ __launch_bounds__(256) void splitk_combine(CombineArgs a) {
  const int64_t total = a.M * a.N;
  for (int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x; t < total;
       t += (int64_t)gridDim.x * 256) {
    const int64_t j = t % a.N;
    float y;
    if (a.split_combine == DG_SEQ) {
      y = a.ws[t];
      for (int s = 1; s < a.S; ++s) {
        y = y + a.ws[(int64_t)s * total + t];
        if (a.merge_bf16) y = round_bf16(y);
      }
    } else {
      // balanced tree over the parts: binary-counter stack, flushed low to high
      float stk[8];
      uint32_t count = 0;
      for (int s = 0; s < a.S; ++s) {
        float v = a.ws[(int64_t)s * total + t];
        uint32_t c = count;
        int lvl = 0;
        while (c & 1u) {
          v = stk[lvl] + v;
          if (a.merge_bf16) v = round_bf16(v);
          c >>= 1;
          ++lvl;
        }
        stk[lvl] = v;
        ++count;
      }
      bool have = false;
      y = 0.f;
      for (int lvl = 0; lvl < 8; ++lvl) {
        if ((count >> lvl) & 1u) {
          if (have) {
            y = stk[lvl] + y;
            if (a.merge_bf16) y = round_bf16(y);
          } else {
            y = stk[lvl];
          }
          have = true;
        }
      }
    }
    float z = y;
    if (a.epilogue != DG_EPI_NONE) z = y + bf16_f32(a.bias[j]);
    if (a.epilogue == DG_EPI_BIAS_SILU) {
      if (a.pre_act) z = round_bf16(z);
      z = silu_f32(z);
    }
    if (a.out_bf16) ((uint16_t*)a.C)[t] = f32_bf16(z);
    else ((float*)a.C)[t] = z;
  }
}

// ----------------------------------------------------------- launchers

hipError_t launch_gemm_generic(const GemmArgs& a, hipStream_t st) {
  dim3 grid((unsigned)((a.N + 15) / 16), (unsigned)((a.M + 15) / 16), (unsigned)a.S);
  hipLaunchKernelGGL(gemm_generic, grid, dim3(64), 0, st, a);
  return hipGetLastError();
}

template <int BM, int BN, int WM, int WN>
static hipError_t launch_tiled_t(const GemmArgs& a, hipStream_t st) {
  dim3 grid((unsigned)((a.N + BN - 1) / BN), (unsigned)((a.M + BM - 1) / BM), (unsigned)a.S);
  hipLaunchKernelGGL((gemm_tiled<BM, BN, WM, WN>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

bool tiled_supported(int tm, int tn) {
  return (tm == 16 && (tn == 64 || tn == 128)) || (tm == 32 && tn == 128) ||
         (tm == 64 && tn == 128) || (tm == 128 && tn == 128);
}

hipError_t launch_gemm_tiled(const GemmArgs& a, int tm, int tn, hipStream_t st) {
  if (tm == 16 && tn == 64) return launch_tiled_t<16, 64, 1, 4>(a, st);
  if (tm == 16 && tn == 128) return launch_tiled_t<16, 128, 1, 4>(a, st);
  if (tm == 32 && tn == 128) return launch_tiled_t<32, 128, 1, 4>(a, st);
  if (tm == 64 && tn == 128) return launch_tiled_t<64, 128, 2, 2>(a, st);
  if (tm == 128 && tn == 128) return launch_tiled_t<128, 128, 2, 2>(a, st);
  return hipErrorInvalidValue;
}

hipError_t launch_splitk_combine(const CombineArgs& a, hipStream_t st) {
  const int64_t total = a.M * a.N;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(splitk_combine, dim3((unsigned)blocks), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace dg
