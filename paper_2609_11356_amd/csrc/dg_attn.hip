// dg_attn.hip -- attention forward for gfx950 whose reduction order is the
// attention descriptor's (paper App. F), independent of the workgroup shape.
//
// Per query row the keys are walked in the descriptor's blocks (width w from
// key 0; under a causal mask the walk splits at the multiples of BLOCK_M:
// the unmasked stage is cut at the query block's start, the masked stage is
// walked from there).  At each block the row's running maximum m, denominator
// l and output row O (binary32) are updated:
//   s_t = RN32(q . k_t * qk_scale)   (+ -1e6 on a masked key above the diagonal)
//   mn = max(m, max_t s_t);  alpha = exp2(m - mn);  p_t = exp2(s_t - mn)
//   l = alpha l + rowsum(p)  (or one fma),  O = alpha O (+) P~ . V
// with P~ = p narrowed to bf16, exp2 the library's own (dg_device.h), the
// block's row sum a chain or the balanced tree over the block's positions,
// and the two matrix multiplications on v_mfma_f32_16x16x32_bf16: the score
// over the head dimension from +0 with the accumulator carried, P~ . V over
// the block's keys from the block start, with alpha O as the accumulator
// (pv_fma) or from +0 and then added.  The end: O / l, or O * (1 / l).
//
// Kernel: one wave per 16 query rows, NW waves per workgroup (the rows of a
// workgroup share one causal split: BLOCK_M is a multiple of 16 NW).  Each
// block's K and V rows go to LDS (zero past the block end, so that a short
// block's missing positions have p = 0 and zero products, which leave every
// accumulator's bits as they are); the wave keeps its Q fragments in
// registers, its S tile and O rows in MFMA accumulators (lane l: rows
// 4 (l / 16) + j, column l % 16), and narrows P through its own LDS area
// into the MFMA operand layout.
#include "dg_device.h"
#include "dg_internal.h"

namespace dg {

namespace {

typedef short shortx8 __attribute__((ext_vector_type(8)));
typedef short shortx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) shortx4* lds_s4;

__device__ __forceinline__ floatx4 mfma(const shortx8& a, const shortx8& b, const floatx4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0,
                                                 0, 0);
}

__device__ __forceinline__ void lds_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// LDS layouts (16-byte chunks; the swizzles only spread a fragment read over
// the banks).  K block [key][dim]: chunk c of key row t at c ^ (t mod DC).
// V block [key][dim] (read transposed): chunk c of key row k at
// c ^ 2 (k mod 4) (^ 8 ((k / 8) mod 2) with 16 chunks a row).  Narrowed P of a
// wave [row][key]: chunk c of row r at c ^ (r mod W/8).
template <int DC>
__device__ __forceinline__ int kofs(int t, int c) {
  return t * DC + (c ^ (t & (DC - 1)));
}
template <int DC>
__device__ __forceinline__ int vofs(int k, int c) {
  if constexpr (DC >= 16) return k * DC + (c ^ ((k & 3) << 1) ^ (((k >> 3) & 1) << 3));
  else return k * DC + (c ^ ((k & 3) << 1));
}
template <int PC>
__device__ __forceinline__ int pofs(int r, int c) {
  return r * PC + (c ^ (r & (PC - 1)));
}

}  // namespace

template <int D, int W, int NW>
__global__ __launch_bounds__(64 * NW) void attn_fwd(AttnArgs a) {
  constexpr int DC = D / 8, PC = W / 8, NST = W / 16, NDT = D / 16, QKS = D / 32, PVS = W / 32;
  static_assert(D % 32 == 0 && W % 32 == 0 && DC >= 8 && PC >= 4, "whole MFMA steps");
  __shared__ __attribute__((aligned(16))) uint16_t Ks[W * D];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[W * D];
  __shared__ __attribute__((aligned(16))) uint16_t Ps[NW][16 * W];
  __shared__ float Fs[NW][16 * (W + 1)];   // the chained block sum: p as binary32, then the row sums

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int li = lane & 15, lg = lane >> 4;
  const int64_t h = blockIdx.y;
  const int64_t r0 = (int64_t)blockIdx.x * (16 * NW);
  const int64_t rw = r0 + 16 * wave;
  const uint16_t* Qh = a.Q + h * a.Lq * D;
  const uint16_t* Kh = a.K + h * a.Lk * D;
  const uint16_t* Vh = a.V + h * a.Lk * D;

  // the wave's Q fragments: row li, head-dimension chunk lg + 4 step
  shortx8 qf[QKS];
  {
    const int64_t i = rw + li;
#pragma unroll
    for (int st = 0; st < QKS; ++st)
      qf[st] = i < a.Lq ? *(const shortx8*)&Qh[i * D + 32 * st + 8 * lg] : shortx8{0, 0, 0, 0, 0, 0, 0, 0};
  }
  int64_t irow[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) irow[j] = rw + 4 * lg + j;

  float m[4], l[4];
  floatx4 O[NDT];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    m[j] = -__builtin_inff();
    l[j] = 0.f;
  }
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) O[dt] = floatx4{0.f, 0.f, 0.f, 0.f};

  // the walk: nb1 unmasked blocks of [0, end1) from key 0, then (causal) nb2
  // masked-stage blocks of [q0, q1) from q0
  int64_t end1 = a.Lk, q0 = 0, q1 = 0;
  if (a.causal) {
    q0 = r0 / a.q_block * a.q_block;
    q1 = q0 + a.q_block < a.Lk ? q0 + a.q_block : a.Lk;
    end1 = q0;
  }
  const int64_t nb1 = (end1 + W - 1) / W, nb2 = a.causal ? (q1 - q0 + W - 1) / W : 0;

  for (int64_t b = 0; b < nb1 + nb2; ++b) {
    const bool masked = b >= nb1;
    const int64_t kb = masked ? q0 + (b - nb1) * W : b * W;
    const int64_t lim = masked ? q1 : end1;
    const int64_t ke = kb + W < lim ? kb + W : lim;

    // the block's K and V rows into LDS (zero past its end)
    __syncthreads();
    for (int q = threadIdx.x; q < W * DC; q += 64 * NW) {
      const int t = q / DC, c = q % DC;
      u32x4 kv = u32x4{0u, 0u, 0u, 0u}, vv = u32x4{0u, 0u, 0u, 0u};
      if (kb + t < ke) {
        kv = *(const u32x4*)&Kh[(kb + t) * D + 8 * c];
        vv = *(const u32x4*)&Vh[(kb + t) * D + 8 * c];
      }
      *(u32x4*)&Ks[8 * kofs<DC>(t, c)] = kv;
      *(u32x4*)&Vs[8 * vofs<DC>(t, c)] = vv;
    }
    __syncthreads();

    // scores: 16 rows x W keys, the head dimension in increasing steps of 32 from +0
    floatx4 S[NST];
#pragma unroll
    for (int st = 0; st < NST; ++st) {
      floatx4 acc = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int k = 0; k < QKS; ++k) {
        const shortx8 kf = *(const shortx8*)&Ks[8 * kofs<DC>(16 * st + li, 4 * k + lg)];
        acc = mfma(qf[k], kf, acc);
      }
      S[st] = acc;
    }

    // scale, mask, block maximum (exact), rescale factor and probabilities
    float bm[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) bm[j] = -__builtin_inff();
#pragma unroll
    for (int st = 0; st < NST; ++st) {
      const int64_t t = kb + 16 * st + li;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float v = S[st][j] * a.qk_scale;
        if (t >= ke) v = -__builtin_inff();
        else if (masked && t > irow[j]) v = v + -1.0e6f;
        S[st][j] = v;
        bm[j] = __builtin_fmaxf(bm[j], v);
      }
    }
    float alpha[4], mn[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) bm[j] = __builtin_fmaxf(bm[j], __shfl_xor(bm[j], o));
      mn[j] = __builtin_fmaxf(m[j], bm[j]);
      alpha[j] = exp2_f32(m[j] - mn[j]);
    }
#pragma unroll
    for (int st = 0; st < NST; ++st)
#pragma unroll
      for (int j = 0; j < 4; ++j) S[st][j] = exp2_f32(S[st][j] - mn[j]);

    // the block's row sums in the descriptor's order
    float rs[4];
    if (a.block_tree) {
      // the perfect tree over the block's W positions in key order (zero past
      // the end: the tree over the live positions): positions 16 st + c of a
      // 16-key sub-tile meet by the lane butterfly xor 1, 2, 4, 8, then the
      // sub-tile roots pairwise
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float sub[NST];
#pragma unroll
        for (int st = 0; st < NST; ++st) {
          float x = S[st][j];
#pragma unroll
          for (int o = 1; o < 16; o <<= 1) x = x + __shfl_xor(x, o);
          sub[st] = x;
        }
#pragma unroll
        for (int w2 = 1; w2 < NST; w2 <<= 1)
#pragma unroll
          for (int st = 0; st < NST; st += 2 * w2) sub[st] = sub[st] + sub[st + w2];
        rs[j] = sub[0];
      }
    } else {
      // the chain in key order: the wave's probabilities through LDS, lane r
      // (r < 16) folds row r, and the roots come back
      float* F = Fs[wave];
#pragma unroll
      for (int st = 0; st < NST; ++st)
#pragma unroll
        for (int j = 0; j < 4; ++j) F[(4 * lg + j) * (W + 1) + 16 * st + li] = S[st][j];
      lds_wait();
      if (lane < 16) {
        float x = F[lane * (W + 1)];
        for (int u = 1; u < W; ++u) x = x + F[lane * (W + 1) + u];
        F[lane * (W + 1) + W] = x;
      }
      lds_wait();
#pragma unroll
      for (int j = 0; j < 4; ++j) rs[j] = F[(4 * lg + j) * (W + 1) + W];
      lds_wait();
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      l[j] = a.l_fma ? __builtin_fmaf(alpha[j], l[j], rs[j]) : alpha[j] * l[j] + rs[j];
      m[j] = mn[j];
    }

    // P narrowed to bf16, into the wave's LDS area in operand layout
    uint16_t* P = Ps[wave];
#pragma unroll
    for (int st = 0; st < NST; ++st)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = 4 * lg + j, u = 16 * st + li;
        P[8 * pofs<PC>(r, u >> 3) + (u & 7)] = f32_bf16(S[st][j]);
      }
    lds_wait();

    // O = alpha O (+) P~ . V over the block's keys from its start
    shortx8 pf[PVS];
#pragma unroll
    for (int k = 0; k < PVS; ++k) pf[k] = *(const shortx8*)&P[8 * pofs<PC>(li, 4 * k + lg)];
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      floatx4 base;
#pragma unroll
      for (int j = 0; j < 4; ++j) base[j] = alpha[j] * O[dt][j];
      floatx4 acc = a.pv_fma ? base : floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int k = 0; k < PVS; ++k) {
        const int n = 16 * dt + 4 * (li & 3);
        const int kr0 = 32 * k + 8 * lg + (li >> 2), kr1 = kr0 + 4;
        const shortx4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)(&Vs[8 * vofs<DC>(kr0, n >> 3) + (n & 7)]));
        const shortx4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)(&Vs[8 * vofs<DC>(kr1, n >> 3) + (n & 7)]));
        const shortx8 vf = shortx8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        acc = mfma(pf[k], vf, acc);
      }
      if (a.pv_fma) O[dt] = acc;
      else
#pragma unroll
        for (int j = 0; j < 4; ++j) O[dt][j] = base[j] + acc[j];
    }
  }

  // the final division (or reciprocal and products), then the output type
  float r[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) r[j] = 1.0f / l[j];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t i = irow[j];
      if (i >= a.Lq) continue;
      const float y = a.final_recip ? O[dt][j] * r[j] : O[dt][j] / l[j];
      const int64_t o = (h * a.Lq + i) * D + 16 * dt + li;
      if (a.out_bf16) ((uint16_t*)a.O)[o] = f32_bf16(y);
      else ((float*)a.O)[o] = y;
    }
}

namespace {

template <int D, int W>
hipError_t launch_dw(const AttnArgs& a, int nw, hipStream_t st) {
  const int64_t rows = 16 * nw;
  dim3 grid((unsigned)((a.Lq + rows - 1) / rows), (unsigned)a.H);
  if (nw == 4) hipLaunchKernelGGL((attn_fwd<D, W, 4>), grid, dim3(256), 0, st, a);
  else if (nw == 2) hipLaunchKernelGGL((attn_fwd<D, W, 2>), grid, dim3(128), 0, st, a);
  else hipLaunchKernelGGL((attn_fwd<D, W, 1>), grid, dim3(64), 0, st, a);
  return hipGetLastError();
}

}  // namespace

bool attn_supported(int64_t d, int key_block) {
  return (d == 64 || d == 128) && (key_block == 32 || key_block == 64 || key_block == 128);
}

hipError_t launch_attention(const AttnArgs& a, int64_t d, int key_block, int nw, hipStream_t st) {
  if (d == 64) {
    if (key_block == 32) return launch_dw<64, 32>(a, nw, st);
    if (key_block == 64) return launch_dw<64, 64>(a, nw, st);
    return launch_dw<64, 128>(a, nw, st);
  }
  if (key_block == 32) return launch_dw<128, 32>(a, nw, st);
  if (key_block == 64) return launch_dw<128, 64>(a, nw, st);
  return launch_dw<128, 128>(a, nw, st);
}

}  // namespace dg
