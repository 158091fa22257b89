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
// Kernel: one wave per RW query rows (16 or 32: one or two 16-row MFMA
// tiles), NW waves per workgroup (the rows of a workgroup share one causal
// split: BLOCK_M is a multiple of RW NW).  Each block's K and V rows are in
// LDS (two buffers: the next block's rows are fetched into registers while
// the current block computes and stored at its end, one barrier per block;
// zero past the block end, so that a short block's missing positions have
// p = 0 and zero products, which leave every accumulator's bits as they
// are).  The wave keeps its Q fragments in registers and its S tile and O
// rows in MFMA accumulators (lane l: rows 4 (l / 16) + j, column l % 16 of a
// 16 x 16 tile).  Score column c of sub-tile st is key NST c + st of the
// block, so the first levels of the block's row-sum tree (key bits below
// NST) are adds within a lane and the last four are DPP lane steps; P~ goes
// through the wave's LDS area as [key][row] (four rows per 8-byte write) and
// comes back in operand layout through the transposing LDS read.
#include "dg_device.h"
#include "dg_internal.h"
#include "dg_lanes.h"

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

// True when alpha[0..3] are 1 on every active lane (one ballot; uniform).
__device__ __forceinline__ bool all_one(const float* alpha) {
  const bool one = alpha[0] == 1.0f && alpha[1] == 1.0f && alpha[2] == 1.0f && alpha[3] == 1.0f;
  return __builtin_amdgcn_ballot_w64(!one) == 0;
}

__device__ __forceinline__ void lds_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

}  // namespace

template <int D, int W, int NW, int RW, bool TREE, bool PF, bool PVF>
__global__ __launch_bounds__(64 * NW) void attn_fwd(AttnArgs a) {
  constexpr int DC = D / 8, NST = W / 16, NDT = D / 16, QKS = D / 32, PVS = W / 32, RT = RW / 16;
  constexpr int LNST = NST == 2 ? 1 : NST == 4 ? 2 : 3;     // log2 NST
  constexpr int PG = RW / 4;                                  // 8-byte groups of a P~ row
  static_assert(D % 32 == 0 && W % 32 == 0 && DC >= 8 && (NST == 2 || NST == 4 || NST == 8), "whole steps");
  constexpr int CHUNKS = W * DC / (64 * NW);                  // K (and V) chunks per thread
  static_assert(!PF || W * DC % (64 * NW) == 0, "whole chunks per thread");
  constexpr int NBUF = PF ? 2 : 1;                            // LDS buffers of K and V
  __shared__ __attribute__((aligned(16))) uint16_t Ks[NBUF][W * D];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[NBUF][W * D];
  __shared__ __attribute__((aligned(16))) uint16_t Ps[NW][W * RW];
  __shared__ float Fs[TREE ? 1 : NW][TREE ? 1 : RW * (W + 1)];   // the chained block sum

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int li = lane & 15, lg = lane >> 4;
  // heads run fastest through the grid, and under a causal mask the query
  // blocks run from the last (the longest walk) to the first
  const int64_t h = blockIdx.x;
  const int64_t qb = a.causal ? (int64_t)gridDim.y - 1 - blockIdx.y : blockIdx.y;
  const int64_t r0 = qb * (RW * NW);
  const int64_t rw = r0 + RW * wave;
  const uint16_t* Qh = a.Q + h * a.Lq * D;
  const uint16_t* Kh = a.K + h * a.Lk * D;
  const uint16_t* Vh = a.V + h * a.Lk * D;

  // K row t: chunk c at c ^ (the row's lane index mod DC), so that the 16
  // rows one fragment read takes land on distinct 16-byte slots
  auto kofs = [](int t, int c) { return t * DC + (c ^ ((t >> LNST) & (DC - 1))); };
  auto vofs = [](int k, int c) {
    if constexpr (DC >= 16) return k * DC + (c ^ ((k & 3) << 1) ^ (((k >> 3) & 1) << 3));
    else return k * DC + (c ^ ((k & 3) << 1));
  };
  // P~ [key u][row r]: 8-byte group g of key row u at g ^ ((u >> LNST) mod PG)
  auto pofs = [](int u, int r) { return u * RW + 4 * ((r >> 2) ^ ((u >> LNST) & (PG - 1))) + (r & 3); };

  shortx8 qf[RT][QKS];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int64_t i = rw + 16 * rt + li;
#pragma unroll
    for (int k = 0; k < QKS; ++k)
      qf[rt][k] = i < a.Lq ? *(const shortx8*)&Qh[i * D + 32 * k + 8 * lg] : shortx8{0, 0, 0, 0, 0, 0, 0, 0};
  }

  float m[RT][4], l[RT][4];
  floatx4 O[RT][NDT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      m[rt][j] = -__builtin_inff();
      l[rt][j] = 0.f;
    }
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) O[rt][dt] = floatx4{0.f, 0.f, 0.f, 0.f};
  }

  // the walk: nb1 unmasked blocks of [0, end1) from key 0, then (causal) nb2
  // masked-stage blocks of [q0, q1) from q0
  int64_t end1 = a.Lk, q0 = 0, q1 = 0;
  if (a.causal) {
    q0 = r0 / a.q_block * a.q_block;
    q1 = q0 + a.q_block < a.Lk ? q0 + a.q_block : a.Lk;
    end1 = q0;
  }
  const int64_t nb1 = (end1 + W - 1) / W, nb = nb1 + (a.causal ? (q1 - q0 + W - 1) / W : 0);
  auto bounds = [&](int64_t b, int64_t* kb, int64_t* ke) {
    const bool st2 = b >= nb1;
    *kb = st2 ? q0 + (b - nb1) * W : b * W;
    const int64_t lim = st2 ? q1 : end1;
    *ke = *kb + W < lim ? *kb + W : lim;
  };
  u32x4 kr[PF ? CHUNKS : 1], vr[PF ? CHUNKS : 1];
  auto fetch = [&](int64_t b) {
    int64_t kb, ke;
    bounds(b, &kb, &ke);
#pragma unroll
    for (int u = 0; u < CHUNKS; ++u) {
      const int q = threadIdx.x + 64 * NW * u, t = q / DC, c = q % DC;
      kr[u] = vr[u] = u32x4{0u, 0u, 0u, 0u};
      if (kb + t < ke) {
        kr[u] = *(const u32x4*)&Kh[(kb + t) * D + 8 * c];
        vr[u] = *(const u32x4*)&Vh[(kb + t) * D + 8 * c];
      }
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int u = 0; u < CHUNKS; ++u) {
      const int q = threadIdx.x + 64 * NW * u, t = q / DC, c = q % DC;
      *(u32x4*)&Ks[buf][8 * kofs(t, c)] = kr[u];
      *(u32x4*)&Vs[buf][8 * vofs(t, c)] = vr[u];
    }
  };
  // without prefetch: the block straight from memory into the one buffer
  auto load_block = [&](int64_t b) {
    int64_t kb, ke;
    bounds(b, &kb, &ke);
    for (int q = threadIdx.x; q < W * DC; q += 64 * NW) {
      const int t = q / DC, c = q % DC;
      u32x4 kv = u32x4{0u, 0u, 0u, 0u}, vv = u32x4{0u, 0u, 0u, 0u};
      if (kb + t < ke) {
        kv = *(const u32x4*)&Kh[(kb + t) * D + 8 * c];
        vv = *(const u32x4*)&Vh[(kb + t) * D + 8 * c];
      }
      *(u32x4*)&Ks[0][8 * kofs(t, c)] = kv;
      *(u32x4*)&Vs[0][8 * vofs(t, c)] = vv;
    }
  };
  if constexpr (PF) {
    if (nb > 0) {
      fetch(0);
      stash(0);
    }
  }

  for (int64_t b = 0; b < nb; ++b) {
    const int cur = PF ? (int)(b & 1) : 0;
    int64_t kb, ke;
    bounds(b, &kb, &ke);
    const bool masked = b >= nb1;
    const bool edge = masked || ke - kb < W;
    __syncthreads();
    if constexpr (PF) {
      if (b + 1 < nb) fetch(b + 1);
    } else {
      load_block(b);
      __syncthreads();
    }
    const uint16_t* K_ = Ks[cur];
    const uint16_t* V_ = Vs[cur];

    // scores: RW rows x W keys (column c of sub-tile st: key NST c + st), the
    // head dimension in increasing steps of 32 from +0; then scaled
    floatx4 S[RT][NST];
#pragma unroll
    for (int st = 0; st < NST; ++st) {
      shortx8 kf[QKS];
#pragma unroll
      for (int k = 0; k < QKS; ++k) kf[k] = *(const shortx8*)&K_[8 * kofs(NST * li + st, 4 * k + lg)];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        floatx4 acc = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int k = 0; k < QKS; ++k) acc = mfma(qf[rt][k], kf[k], acc);
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[j] = acc[j] * a.qk_scale;
        S[rt][st] = acc;
      }
    }
    // positions past the block end drop out (-inf), masked keys get -1e6
    if (edge) {
#pragma unroll
      for (int st = 0; st < NST; ++st) {
        const int64_t t = kb + NST * li + st;
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int64_t i = rw + 16 * rt + 4 * lg + j;
            float v = S[rt][st][j];
            if (t >= ke) v = -__builtin_inff();
            else if (masked && t > i) v = v + -1.0e6f;
            S[rt][st][j] = v;
          }
      }
    }

#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      float alpha[4], rs[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float bm = S[rt][0][j];
#pragma unroll
        for (int st = 1; st < NST; ++st) bm = __builtin_fmaxf(bm, S[rt][st][j]);
        bm = max_lanes<4>(bm);
        const float mn = __builtin_fmaxf(m[rt][j], bm);
        alpha[j] = exp2_f32(m[rt][j] - mn);
        m[rt][j] = mn;
#pragma unroll
        for (int st = 0; st < NST; ++st) S[rt][st][j] = exp2_f32(S[rt][st][j] - mn);
      }
      if constexpr (TREE) {
        // the perfect tree over the block's positions in key order: key bits
        // below NST within the lane, then the 16 lanes of the row group
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          float v[NST];
#pragma unroll
          for (int st = 0; st < NST; ++st) v[st] = S[rt][st][j];
#pragma unroll
          for (int w2 = 1; w2 < NST; w2 <<= 1)
#pragma unroll
            for (int st = 0; st < NST; st += 2 * w2) v[st] = v[st] + v[st + w2];
          rs[j] = tree_sum_lanes<4>(v[0]);
        }
      } else {
        // the chain in key order through the wave's LDS area
        float* F = Fs[wave];
#pragma unroll
        for (int st = 0; st < NST; ++st)
#pragma unroll
          for (int j = 0; j < 4; ++j) F[(16 * rt + 4 * lg + j) * (W + 1) + NST * li + st] = S[rt][st][j];
        lds_wait();
        if (lane < 16) {
          const float* row = &F[(16 * rt + lane) * (W + 1)];
          float x = row[0];
          for (int u = 1; u < W; ++u) x = x + row[u];
          F[(16 * rt + lane) * (W + 1) + W] = x;
        }
        lds_wait();
#pragma unroll
        for (int j = 0; j < 4; ++j) rs[j] = F[(16 * rt + 4 * lg + j) * (W + 1) + W];
        lds_wait();
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) l[rt][j] = a.l_fma ? __builtin_fmaf(alpha[j], l[rt][j], rs[j]) : alpha[j] * l[rt][j] + rs[j];

      // P~ = p narrowed to bf16 into the wave's [key][row] area, four rows per write
      uint16_t* P = Ps[wave];
#pragma unroll
      for (int st = 0; st < NST; ++st) {
        const int u = NST * li + st;
        const uint32_t lo = f32x2_bf16x2(S[rt][st][0], S[rt][st][1]), hi = f32x2_bf16x2(S[rt][st][2], S[rt][st][3]);
        *(uint2*)&P[pofs(u, 16 * rt + 4 * lg)] = uint2{lo, hi};
      }
      // rescale the output rows (skipped when every row of the wave keeps its
      // maximum: alpha = 1 and 1 x O = O exactly)
      if (!all_one(alpha))
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
          for (int j = 0; j < 4; ++j) O[rt][dt][j] = alpha[j] * O[rt][dt][j];
    }
    lds_wait();

    // O = alpha O (+) P~ . V over the block's keys from its start, for each
    // output element the steps of 32 keys in increasing order
    const uint16_t* P = Ps[wave];
    shortx8 pf[RT][PVS];
#pragma unroll
    for (int k = 0; k < PVS; ++k)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const int n = 16 * rt + 4 * (li & 3);
        const int u0 = 32 * k + 8 * lg + (li >> 2), u1 = u0 + 4;
        const shortx4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)(&P[pofs(u0, n)]));
        const shortx4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)(&P[pofs(u1, n)]));
        pf[rt][k] = shortx8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      }
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      floatx4 acc[RT];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) acc[rt] = PVF ? O[rt][dt] : floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int k = 0; k < PVS; ++k) {
        const int n = 16 * dt + 4 * (li & 3);
        const int kr0 = 32 * k + 8 * lg + (li >> 2), kr1 = kr0 + 4;
        const shortx4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)(&V_[8 * vofs(kr0, n >> 3) + (n & 7)]));
        const shortx4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)(&V_[8 * vofs(kr1, n >> 3) + (n & 7)]));
        const shortx8 vf = shortx8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) acc[rt] = mfma(pf[rt][k], vf, acc[rt]);
      }
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        if constexpr (PVF) O[rt][dt] = acc[rt];
        else
#pragma unroll
          for (int j = 0; j < 4; ++j) O[rt][dt][j] = O[rt][dt][j] + acc[rt][j];
      }
    }
    if constexpr (PF) {
      if (b + 1 < nb) stash(cur ^ 1);
    }
  }

  // the final division (or reciprocal and products), then the output type
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    float r[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) r[j] = 1.0f / l[rt][j];
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int64_t i = rw + 16 * rt + 4 * lg + j;
        if (i >= a.Lq) continue;
        const float y = a.final_recip ? O[rt][dt][j] * r[j] : O[rt][dt][j] / l[rt][j];
        const int64_t o = (h * a.Lq + i) * D + 16 * dt + li;
        if (a.out_bf16) ((uint16_t*)a.O)[o] = f32_bf16(y);
        else ((float*)a.O)[o] = y;
      }
  }
}

namespace {

template <int D, int W, int NW, int RW, bool PF>
hipError_t launch_one(const AttnArgs& a, hipStream_t st) {
  constexpr int rows = NW * RW;
  dim3 grid((unsigned)a.H, (unsigned)((a.Lq + rows - 1) / rows));
  const dim3 blk(64 * NW);
  if (a.block_tree) {
    if (a.pv_fma) hipLaunchKernelGGL((attn_fwd<D, W, NW, RW, true, PF, true>), grid, blk, 0, st, a);
    else hipLaunchKernelGGL((attn_fwd<D, W, NW, RW, true, PF, false>), grid, blk, 0, st, a);
  } else {
    if (a.pv_fma) hipLaunchKernelGGL((attn_fwd<D, W, NW, RW, false, PF, true>), grid, blk, 0, st, a);
    else hipLaunchKernelGGL((attn_fwd<D, W, NW, RW, false, PF, false>), grid, blk, 0, st, a);
  }
  return hipGetLastError();
}

// Workgroup shape (speed only): 16-row waves (registers), eight of them
// with the next block prefetched into a second buffer when the causal split
// allows 128-row workgroups (four when it allows 64), else fewer waves
// loading each block as it comes.  Measured on MI355X at 32 x 4096 x 128:
// eight 16-row waves 357 TFLOP/s against 268 for four 32-row waves.
template <int D, int W>
hipError_t launch_dw(const AttnArgs& a, hipStream_t st) {
  const int64_t bm = a.causal ? a.q_block : 128;
  if constexpr (W == 128) {
    if (bm % 64 == 0) return launch_one<D, W, 4, 16, false>(a, st);
    return launch_one<D, W, 1, 16, false>(a, st);
  } else {
    // prefetch needs whole 16-byte chunks of the block per thread
    constexpr bool pf8 = W * (D / 8) % 512 == 0, pf4 = W * (D / 8) % 256 == 0;
    if (bm % 128 == 0) return launch_one<D, W, 8, 16, pf8>(a, st);
    if (bm % 64 == 0) return launch_one<D, W, 4, 16, pf4>(a, st);
    if (bm % 32 == 0) return launch_one<D, W, 2, 16, false>(a, st);
    return launch_one<D, W, 1, 16, false>(a, st);
  }
}

}  // namespace

bool attn_supported(int64_t d, int key_block) {
  return (d == 64 || d == 128) && (key_block == 32 || key_block == 64 || key_block == 128);
}

hipError_t launch_attention(const AttnArgs& a, int64_t d, int key_block, hipStream_t st) {
  if (d == 64) {
    if (key_block == 32) return launch_dw<64, 32>(a, st);
    if (key_block == 64) return launch_dw<64, 64>(a, st);
    return launch_dw<64, 128>(a, st);
  }
  if (key_block == 32) return launch_dw<128, 32>(a, st);
  if (key_block == 64) return launch_dw<128, 64>(a, st);
  return launch_dw<128, 128>(a, st);
}

}  // namespace dg
