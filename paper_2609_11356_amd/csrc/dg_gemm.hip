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
#include <mutex>
#include <type_traits>

#include "dg_device.h"
#include "dg_internal.h"
#include "dg_mma.h"

// Split-K partials of dg_gemm_noalloc: a fixed array, one copy per device,
// held until the process ends.  Host code never uses this name as an address
// (on the host it only stands for the symbol); it asks the runtime for each
// device's copy once (noalloc_scratch) and passes that pointer to the kernels.
static __device__ __align__(256) float scratch[DG_NOALLOC_SCRATCH_BYTES / sizeof(float)];

namespace dg {

hipError_t noalloc_scratch(void** out) {
  static std::mutex mu;
  static void* addr[64];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *out = addr[dev];
  return hipSuccess;
}


// Sixteen zero bytes (device globals start zeroed).  A load that falls
// outside the matrix or past the part end reads this instead, so that no
// instruction touches a loaded value before it is stored -- a select on the
// loaded value would make the load wait at once.
__device__ u32x4 g_zero16[1];

__device__ __forceinline__ const u32x4* chunk_or_zero(bool ok, const uint16_t* p) {
  return ok ? reinterpret_cast<const u32x4*>(p) : &g_zero16[0];
}

// LDS layout of A slabs ([row][k], CPR 16-byte chunks per row): chunk c of
// row r sits at position c ^ swz_a<CPR>(r).  A fragment read takes one chunk
// of 16 consecutive rows; with 64-byte rows (CPR 4) the swizzle gives every
// 8 consecutive rows distinct 16-byte slots of a 128-byte bank window and
// every 16 rows distinct slots of a 256-byte one (with 128-byte rows, CPR 8,
// likewise one row per 128 bytes), so the read has no bank conflict whether
// the LDS serves 8 or 16 lanes per pass.  Measured on the MLP kernel: bank
// conflict cycles fell from 1.7e7 to 4.6e5 and the kernel's cycles by 9 %
// against the earlier swizzle c ^ ((r / 4) mod 4).
template <int CPR>
__device__ __forceinline__ int swz_a(int row) {
  static_assert(CPR == 4 || CPR == 8, "64- or 128-byte rows");
  constexpr int sh = CPR == 4 ? 1 : 0;
  return ((row >> sh) ^ (row >> (sh + 1))) & (CPR - 1);
}



// An operand as binary32 (exact for both formats).
template <bool F16>
__device__ __forceinline__ float op_f32(uint16_t h) {
  if constexpr (F16) return (float)__builtin_bit_cast(_Float16, h);
  else return bf16_f32(h);
}

// The same instruction with the accumulator tied to one accumulation
// register quad (input and output the same registers), for kernels whose
// accumulators fill that register file: the compiler otherwise renames
// accumulators between loop iterations and copies them back.  The compiler
// does not see an MFMA here, so a reader of the accumulator through another
// instruction must first wait for the last one to finish (mfma_drain).
__device__ __forceinline__ void mfma16_tied(floatx4& acc, const shortx8& a, const shortx8& b) {
  asm("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}

// Wait states after an MFMA before its result is read by a non-MFMA
// instruction (more than the 16x16x32 instruction's latency).
__device__ __forceinline__ void mfma_drain() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}


// finish() for four consecutive columns j..j+3 (all < N: the tiled path
// requires N % 8 == 0 and 16-byte aligned C), with one vector store; b4 holds
// the bias of those columns as binary32 (used only by the epilogue).  Returns
// the four values as stored in C, as binary32 (the partials when S > 1).
__device__ __forceinline__ float4 finish4v(const GemmArgs& a, int s, int64_t i, int64_t j, float4 y4, float4 b4) {
  float y[4] = {y4.x, y4.y, y4.z, y4.w};
#pragma unroll
  for (int e = 0; e < 4; ++e)
    if (a.partial_bf16) y[e] = round_bf16(y[e]);
  if (a.S > 1) {
    *(float4*)&a.ws[((int64_t)s * a.M + i) * a.N + j] = float4{y[0], y[1], y[2], y[3]};
    return float4{y[0], y[1], y[2], y[3]};
  }
  if (a.epilogue != DG_EPI_NONE) {
    const float b[4] = {b4.x, b4.y, b4.z, b4.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) y[e] = y[e] + b[e];
  }
  if (a.epilogue == DG_EPI_BIAS_SILU) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float z = y[e];
      if (a.pre_act) z = round_bf16(z);
      y[e] = silu_f32(z);
    }
  }
  if (a.out_bf16) {
    const uint32_t lo = f32x2_bf16x2(y[0], y[1]);
    const uint32_t hi = f32x2_bf16x2(y[2], y[3]);
    *(uint2*)&((uint16_t*)a.C)[i * a.N + j] = uint2{lo, hi};
    return float4{bits_f32(lo << 16), bits_f32(lo & 0xffff0000u), bits_f32(hi << 16), bits_f32(hi & 0xffff0000u)};
  }
  *(float4*)&((float*)a.C)[i * a.N + j] = float4{y[0], y[1], y[2], y[3]};
  return float4{y[0], y[1], y[2], y[3]};
}

// finish4v with the bias read from memory.
__device__ __forceinline__ void finish4(const GemmArgs& a, int s, int64_t i, int64_t j, float4 y4) {
  float4 b4 = float4{0.f, 0.f, 0.f, 0.f};
  if (a.S == 1 && a.epilogue != DG_EPI_NONE) {
    const uint2 bb = *(const uint2*)&a.bias[j];
    b4 = float4{bits_f32(bb.x << 16), bits_f32(bb.x & 0xffff0000u), bits_f32(bb.y << 16), bits_f32(bb.y & 0xffff0000u)};
  }
  (void)finish4v(a, s, i, j, y4, b4);
}

// Whether the epilogue reads the bias (a single part, bias epilogue).
__device__ __forceinline__ bool needs_bias(const GemmArgs& a) { return a.S == 1 && a.epilogue != DG_EPI_NONE; }

// The bias of columns [j0, j0 + n) as binary32 into LDS (zero past N), by
// all threads of the workgroup; the caller synchronises afterwards.
__device__ __forceinline__ void stage_bias(const GemmArgs& a, int64_t j0, int n, float* bsh) {
  if (!needs_bias(a)) return;
  for (int c = threadIdx.x; c < n; c += blockDim.x) bsh[c] = j0 + c < a.N ? bf16_f32(a.bias[j0 + c]) : 0.f;
}

// Wait for the wave's own LDS operations (and keep the compiler from moving
// memory operations across).  LDS operations of one wave run in issue order,
// so after this a read sees what the wave wrote before.
__device__ __forceinline__ void lds_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// Epilogue of one wave's (16 TM) x (16 TN) tile of 16x16 MFMA accumulators
// (lane l holds rows 4 (l / 16) .. +3, column l % 16 of each), rows from ib
// and columns from jb.  Each 16-row band passes through the wave's own LDS
// area cs (16 rows of pitch 16 TN + 4 floats: rows 4 apart start 16 banks
// apart) and leaves as four-column vectors; the bias of the wave's columns
// comes from bsh (staged by stage_bias), so no global load waits inside the
// loop.  Only the wave itself touches cs, so no workgroup barrier is needed.
// With croot set, the wave also folds each of its columns down its 16 TM
// rows as the perfect tree of the values stored in C (rows past M count as
// -0, the exact identity): the band's values go back into cs, lane c takes
// column c of the band (rows paired from the top, 16-row band roots paired
// the same way), and the root lands in croot[c].
template <int TM, int TN, typename Acc>
__device__ __forceinline__ void wave_epilogue(const GemmArgs& a, int s, int64_t ib, int64_t jb, float* cs,
                                              const float* bsh, const Acc& acc, float* croot = nullptr) {
  constexpr int WTN = 16 * TN, CSP = WTN + 4;
  static_assert((TM & (TM - 1)) == 0, "a power-of-two band count");
  const int lane = threadIdx.x & 63;
  const bool bias = needs_bias(a), tree = WTN <= 64 && croot != nullptr;   // one column per lane
  float band[TM];
#pragma unroll
  for (int mi = 0; mi < TM; ++mi) {
#pragma unroll
    for (int ni = 0; ni < TN; ++ni)
#pragma unroll
      for (int r = 0; r < 4; ++r) cs[(4 * (lane >> 4) + r) * CSP + 16 * ni + (lane & 15)] = acc[mi][ni][r];
    lds_wait();
#pragma unroll 1
    for (int q = lane; q < 16 * WTN / 4; q += 64) {
      const int rr = q / (WTN / 4), cc = 4 * (q % (WTN / 4));
      const int64_t i = ib + 16 * mi + rr, j = jb + cc;
      float4* p = (float4*)&cs[rr * CSP + cc];
      const float4 y4 = *p;
      const float4 b4 = bias ? *(const float4*)&bsh[cc] : float4{0.f, 0.f, 0.f, 0.f};
      float4 v = float4{-0.f, -0.f, -0.f, -0.f};
      if (i < a.M && j < a.N) v = finish4v(a, s, i, j, y4, b4);
      if (tree) *p = v;
    }
    lds_wait();
    if (WTN <= 64 && tree) {
      float v[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) v[r] = lane < WTN ? cs[r * CSP + lane] : 0.f;
#pragma unroll
      for (int w = 1; w < 16; w <<= 1)
#pragma unroll
        for (int r = 0; r < 16; r += 2 * w) v[r] = v[r] + v[r + w];
      band[mi] = v[0];
      lds_wait();
    }
  }
  if (WTN <= 64 && tree) {
#pragma unroll
    for (int w = 1; w < TM; w <<= 1)
#pragma unroll
      for (int mi = 0; mi < TM; mi += 2 * w) band[mi] = band[mi] + band[mi + w];
    if (lane < WTN) croot[lane] = band[0];
  }
}

// --------------------------------------------- scalar path (chained chunks)
//
// The descriptor with the scalar instruction (groups of one product, each
// joining the accumulator by one fused multiply-add: the scalar path of
// Sec. 3.2.2, where a chunk of the axis is an explicit FMA chain).  One
// thread per output column and part, MR rows at once; the part's positions
// are walked in order (contiguous part, or the dealt tiles of a strided
// split), in windows whose A values the workgroup stages in LDS (every
// thread reads the same value: a broadcast); accumulator tiles close every
// tile_k positions from the part start (a short first tile when tail-first)
// and are carried, chained or met in the balanced tree.  No MFMA row waste:
// the shape of choice for one or a few rows split over many chunks.
template <int MR, int CPT, bool F16>
__global__ __launch_bounds__(256) void gemm_scalar(GemmArgs a) {
  constexpr int W = 256;                  // positions per staged window
  constexpr int U = 16;                   // positions whose loads are in flight together
  __shared__ __attribute__((aligned(16))) float As[MR][W];
  const int64_t j = ((int64_t)blockIdx.x * 256 + threadIdx.x) * CPT;   // first of CPT columns
  const bool col = j < a.N;
  const int64_t i0 = (int64_t)blockIdx.y * MR;
  const int s = blockIdx.z;
  const int64_t tk = a.tile_k, w = a.split_w, K = a.K;
  const bool strided = w != 0;
  // positions of the part
  int64_t len;
  if (strided) {
    len = 0;
    for (int64_t u = s; u * w < K; u += a.S) len += (K - u * w < w) ? K - u * w : w;
  } else {
    len = a.cuts[s + 1] - a.cuts[s];
  }
  auto kpos = [&](int64_t q) -> int64_t {
    return strided ? (s + a.S * (q / w)) * w + q % w : a.cuts[s] + q;
  };
  const int64_t off = (!strided && a.tail_first) ? len % tk : 0;   // short first tile
  auto next_start = [&](int64_t q) -> int64_t {                     // first tile start after q
    if (off > 0 && q < off) return off;
    return off + ((q - off) / tk + 1) * tk;
  };
  // CPT consecutive columns of row k of B (zero past N)
  auto bload = [&](int64_t k, float* v) {
    const uint16_t* bp = a.B + k * a.N + j;
    if constexpr (CPT == 4) {
      const uint2 q = col ? *(const uint2*)bp : uint2{0u, 0u};
      v[0] = op_f32<F16>((uint16_t)q.x); v[1] = op_f32<F16>((uint16_t)(q.x >> 16));
      v[2] = op_f32<F16>((uint16_t)q.y); v[3] = op_f32<F16>((uint16_t)(q.y >> 16));
    } else {
      v[0] = col ? op_f32<F16>(bp[0]) : 0.0f;
    }
  };
  float acc[MR][CPT], part[MR][CPT], st[MR][CPT][32];
#pragma unroll
  for (int r = 0; r < MR; ++r)
#pragma unroll
    for (int c = 0; c < CPT; ++c) acc[r][c] = part[r][c] = 0.0f;
  bool have = false;
  uint32_t count = 0;
  auto push = [&](float v, int r, int c) {
    int l = 0;
    for (uint32_t cc = count; cc & 1u; cc >>= 1) v = st[r][c][l++] + v;
    st[r][c][l] = v;
  };
  auto close = [&]() {
    if (a.tile_combine == DG_CARRY) return;
#pragma unroll
    for (int r = 0; r < MR; ++r)
#pragma unroll
      for (int c = 0; c < CPT; ++c) {
        if (a.tile_combine == DG_SEQ) part[r][c] = have ? part[r][c] + acc[r][c] : acc[r][c];
        else push(acc[r][c], r, c);
        acc[r][c] = 0.0f;
      }
    have = true;
    ++count;
  };
  for (int64_t w0 = 0; w0 < len; w0 += W) {
    const int n = (int)((len - w0 < W) ? len - w0 : W);
    __syncthreads();   // the previous window has been read
    for (int e = threadIdx.x; e < MR * W; e += 256) {
      const int r = e / W, qq = e % W;
      As[r][qq] = (qq < n && i0 + r < a.M) ? op_f32<F16>(a.A[(i0 + r) * K + kpos(w0 + qq)]) : 0.0f;
    }
    __syncthreads();
    int qq = 0;
    while (qq < n) {
      const int64_t q = w0 + qq;
      if (q != 0 && (q == off || (q > off && (q - off) % tk == 0))) close();
      const int64_t nx = next_start(q);
      const int end = (int)((nx - w0 < n) ? nx - w0 : n);
      // positions [qq, end) lie in one tile and one dealt tile: consecutive k
      const int64_t kq = kpos(q);
      const int cnt = end - qq;
      int t = 0;
      for (; t + U <= cnt; t += U) {
        float bv[U][CPT];
#pragma unroll
        for (int e = 0; e < U; ++e) bload(kq + t + e, bv[e]);
#pragma unroll
        for (int e = 0; e < U; ++e)
#pragma unroll
          for (int r = 0; r < MR; ++r) {
            const float av = As[r][qq + t + e];
#pragma unroll
            for (int c = 0; c < CPT; ++c) acc[r][c] = __builtin_fmaf(av, bv[e][c], acc[r][c]);
          }
      }
      for (; t < cnt; ++t) {
        float bv[CPT];
        bload(kq + t, bv);
#pragma unroll
        for (int r = 0; r < MR; ++r)
#pragma unroll
          for (int c = 0; c < CPT; ++c) acc[r][c] = __builtin_fmaf(As[r][qq + t], bv[c], acc[r][c]);
      }
      qq = end;
    }
  }
  // the part's value: the last tile joins as every other did
#pragma unroll
  for (int r = 0; r < MR; ++r)
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      float pv;
      if (a.tile_combine == DG_CARRY || len == 0) {
        pv = acc[r][c];
      } else if (a.tile_combine == DG_SEQ) {
        pv = have ? part[r][c] + acc[r][c] : acc[r][c];
      } else {
        push(acc[r][c], r, c);
        const uint32_t cnt2 = count + 1;
        float res = 0.0f;
        bool h = false;
        for (int lv = 0; lv < 32; ++lv)
          if ((cnt2 >> lv) & 1u) {
            res = h ? st[r][c][lv] + res : st[r][c][lv];
            h = true;
          }
        pv = res;
      }
      if (col && i0 + r < a.M && j + c < a.N) finish(a, s, i0 + r, j + c, pv);
    }
}

// The fp8 instructions (OCP e4m3 operands).  16x16x32: lane l holds 8 bytes,
// k = 8(l/16) + e.  The block-scaled 16x16x128 (format 0 = e4m3 for both
// operands, E8M0 scales 127 = 1.0): 32 bytes, bytes 0..15 at
// k = 16(l/16) + e and bytes 16..31 at k = 64 + 16(l/16) + e.  Both fold
// the same chain of 16-k chunks.
typedef int intx8 __attribute__((ext_vector_type(8)));
typedef int intx2 __attribute__((ext_vector_type(2)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
__device__ __forceinline__ floatx4 mfma_fp8(uint64_t a, uint64_t b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_fp8_fp8((long)a, (long)b, c, 0, 0, 0);
}
__device__ __forceinline__ floatx4 mfma_fp8x128(const intx8& a, const intx8& b, const floatx4& c) {
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 0, 0, 127, 0, 127);
}

// ------------------------------------------------------------- generic

__global__ __launch_bounds__(64) void gemm_generic(GemmArgs a) {
  __shared__ floatx4 stk[32][64];  // binary-counter stack for the tile tree
  const int lane = threadIdx.x;
  const int64_t i0 = (int64_t)blockIdx.y * 16, j0 = (int64_t)blockIdx.x * 16;
  const int s = blockIdx.z;
  const int64_t tk = a.tile_k;
  const int64_t arow = i0 + (lane & 15), bcol = j0 + (lane & 15);
  const int kb = 8 * (lane >> 4);
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
  const int64_t step = a.fma ? 32 : a.group;  // one instruction per step
  floatx4 acc = zero;
  uint32_t count = 0;
  int64_t t = 0;  // tiles of the part so far
  // one accumulator tile [ts, te) of the part
  auto tile = [&](int64_t ts, int64_t te) {
    floatx4 v = (a.tile_combine == DG_CARRY) ? acc : zero;
    for (int64_t gs = ts; gs < te; gs += step) {
      const int64_t ge = (gs + step < te) ? gs + step : te;
      if (a.ab_e4m3) {
        // e4m3 x e4m3: the group's 32-k instructions chained from the
        // accumulator (fma = 1) or from +0 (fma = 0); a 16-k group is one
        // instruction whose second chunk is empty, which leaves it as it is
        floatx4 w = a.fma ? v : zero;
        for (int64_t ss = gs; ss < ge; ss += 32) {
          uint64_t av8 = 0, bv8 = 0;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int64_t k = ss + kb + e;
            const bool ok = k < ge;
            const uint64_t x = (ok && arow < a.M) ? ((const uint8_t*)a.A)[arow * a.K + k] : 0;
            const uint64_t y = (ok && bcol < a.N) ? ((const uint8_t*)a.B)[k * a.N + bcol] : 0;
            av8 |= x << (8 * e);
            bv8 |= y << (8 * e);
          }
          w = mfma_fp8(av8, bv8, w);
        }
        v = a.fma ? w : v + w;
        continue;
      }
      shortx8 av, bv;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int64_t k = gs + kb + e;
        const bool ok = k < ge;
        av[e] = (ok && arow < a.M) ? (short)a.A[arow * a.K + k] : (short)0;
        if (a.b_e4m3)
          bv[e] = (ok && bcol < a.N) ? (short)e4m3_bf16(((const uint8_t*)a.B)[k * a.N + bcol]) : (short)0;
        else
          bv[e] = (ok && bcol < a.N) ? (short)a.B[k * a.N + bcol] : (short)0;
      }
      if (a.fma) {
        v = a.in_f16 ? mfma16h(av, bv, v) : mfma16(av, bv, v);
      } else {
        floatx4 w = a.in_f16 ? mfma16h(av, bv, zero) : mfma16(av, bv, zero);
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
    ++t;
  };
  if (a.split_w == 0) {
    // contiguous part [cuts[s], cuts[s+1]): tiles of tile_k from its start,
    // the short one first or last
    const int64_t k0 = a.cuts[s], k1 = a.cuts[s + 1];
    const int64_t len = k1 - k0;
    const int64_t ntiles = (len + tk - 1) / tk;
    int64_t first = tk;
    if (a.tail_first && (len % tk)) first = len % tk;
    int64_t ts = k0;
    for (int64_t u = 0; u < ntiles; ++u) {
      int64_t tl = (u == 0) ? (first < len ? first : len) : tk;
      if (ts + tl > k1) tl = k1 - ts;
      tile(ts, ts + tl);
      ts += tl;
    }
  } else {
    // strided part: dealt tiles u = s, s + S, ... of width w, each cut into
    // accumulator tiles of tile_k (w is a multiple of tile_k)
    const int64_t w = a.split_w;
    for (int64_t u = s; u * w < a.K; u += a.S) {
      const int64_t ue = (u * w + w < a.K) ? u * w + w : a.K;
      for (int64_t ts = u * w; ts < ue; ts += tk) tile(ts, (ts + tk < ue) ? ts + tk : ue);
    }
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

// A 16-byte vector of A row `row` at k..k+7, zero past M or past the part
// end (the tiled paths run only where part ends are multiples of 8, so a
// vector is wholly inside or wholly outside).
__device__ __forceinline__ u32x4 load_a_vec(const GemmArgs& a, int64_t row, int64_t k, int64_t k1) {
  return *chunk_or_zero(row < a.M && k < k1, a.A + row * a.K + k);
}

// A 16-byte vector of B row k at columns n..n+7 (N % 8 == 0: all or none).
__device__ __forceinline__ u32x4 load_b_vec(const GemmArgs& a, int64_t k, int64_t n, int64_t k1) {
  return *chunk_or_zero(k < k1 && n < a.N, a.B + k * a.N + n);
}

template <int BM, int BN, int WM, int WN>
__device__ __forceinline__ void tiled_body(const GemmArgs& a, int64_t i0, int64_t j0) {
  static_assert(WM * WN == 4, "four waves");
  constexpr int WTM = BM / WM, WTN = BN / WN;  // rows / cols per wave
  constexpr int TM = WTM / 16, TN = WTN / 16;  // 16x16 MFMA blocks per wave
  static_assert(TM >= 1 && TN >= 1 && WTM % 16 == 0 && WTN % 16 == 0, "wave tile");
  constexpr int AV = BM * (BK / 8);            // 16 B vectors in an A slab
  constexpr int BB = (BK / 4) * (BN / 8);      // 4x8 blocks in a B slab
  constexpr int AV_T = (AV + 255) / 256, BB_T = (BB + 255) / 256;

  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * (BM + BN) * LDS_PITCH];
  uint16_t (*As)[BM][LDS_PITCH] = reinterpret_cast<uint16_t (*)[BM][LDS_PITCH]>(smem);
  uint16_t (*Bs)[BN][LDS_PITCH] = reinterpret_cast<uint16_t (*)[BN][LDS_PITCH]>(smem + 2 * BM * LDS_PITCH);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int s = blockIdx.z;
  const int64_t k0 = a.cuts[s], k1 = a.cuts[s + 1];
  const int nslab = (int)((k1 - k0 + BK - 1) / BK);

  floatx4 acc[TM][TN];
#pragma unroll
  for (int mi = 0; mi < TM; ++mi)
#pragma unroll
    for (int ni = 0; ni < TN; ++ni) acc[mi][ni] = floatx4{0.f, 0.f, 0.f, 0.f};

  u32x4 ra[AV_T];
  u32x4 rb[BB_T][4];

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
        *(u32x4*)&As[buf][v / (BK / 8)][8 * (v % (BK / 8))] = ra[t];
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

  // Epilogue through LDS, one 16-row strip of every wave at a time: the
  // accumulators are parked as fp32, then each lane finishes 4 consecutive
  // columns (bias, SiLU, rounding) and stores them with one vector store.
  // staging rows of pitch WTN + 4 floats: the four row groups a write
  // instruction covers (rows 4 apart) start 16 banks apart
  constexpr int CSP = WTN + 4;
  float* cs = reinterpret_cast<float*>(smem) + wave * 16 * CSP;
  static_assert(4 * 16 * CSP * 4 <= (int)sizeof(smem), "epilogue staging fits");
#pragma unroll
  for (int mi = 0; mi < TM; ++mi) {
    __syncthreads();
#pragma unroll
    for (int ni = 0; ni < TN; ++ni)
#pragma unroll
      for (int r = 0; r < 4; ++r) cs[(4 * (lane >> 4) + r) * CSP + 16 * ni + (lane & 15)] = acc[mi][ni][r];
    __syncthreads();
#pragma unroll 1
    for (int q = lane; q < 16 * WTN / 4; q += 64) {
      const int rr = q / (WTN / 4), cc = 4 * (q % (WTN / 4));
      const int64_t i = i0 + wm * WTM + 16 * mi + rr, j = j0 + wn * WTN + cc;
      if (i < a.M && j < a.N) finish4(a, s, i, j, *(const float4*)&cs[rr * CSP + cc]);
    }
  }
}

// Blocks of up to 128x128: several workgroups per CU.
template <int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(256) void gemm_tiled(GemmArgs a) {
  tiled_body<BM, BN, WM, WN>(a, (int64_t)blockIdx.y * BM, (int64_t)blockIdx.x * BN);
}

// 256-wide blocks: one workgroup per CU, one wave per SIMD, so that a wave
// may hold its 128x128 (or 128x64) accumulator tile in the AGPR file next to
// the staging registers.  Tiles are visited in groups of eight block rows,
// column by column, so concurrently running workgroups share B panels.
template <int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void gemm_big(GemmArgs a) {
  const int tiles_m = (int)((a.M + BM - 1) / BM);
  const int w = blockIdx.x;
  constexpr int GROUP = 8;
  const int tiles_n = gridDim.x / tiles_m;
  const int group = w / (GROUP * tiles_n);
  const int first = group * GROUP;
  const int rows = (tiles_m - first < GROUP) ? tiles_m - first : GROUP;
  const int in_group = w - group * GROUP * tiles_n;
  const int ty = first + in_group % rows, tx = in_group / rows;
  tiled_body<BM, BN, WM, WN>(a, (int64_t)ty * BM, (int64_t)tx * BN);
}

// ------------------------------------------------------------ tiled v3
//
// Same order as gemm_tiled (16x16x32 MFMA chain, 8-k chunks from k = 0), with
// a deeper, branch-free pipeline:
//   * A and B live in LDS in their global row-major layouts ([m][k], [k][n]),
//     16-byte chunks XOR-swizzled per row so that fragment reads spread over
//     the banks; B fragments come out of LDS already transposed through
//     ds_read_b64_tr_b16 (a 16-lane group reading rows k0..k0+3, 4 columns
//     per lane, hands lane j column j of those 4 rows);
//   * every chunk is either wholly inside the part and the matrix or wholly
//     outside (part ends and N are multiples of 8), so a load is a select
//     between a 16-byte load and zero, with no branches;
//   * global loads run two 64-k slabs ahead through a ring of two register
//     sets, into an LDS double buffer, one barrier per slab.
typedef short shortx4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) shortx4* lds_s4;

// The same pipeline serves the descriptors whose accumulator is not one
// carried chain (tile_combine chain or tree, or fma = 0) when every tile
// boundary lies on a 32-k step from the part start: COMB is the tile
// combine, FMA0 that each 32-k instruction starts from zero and its result
// is added to the tile's accumulator (v = v + w, one binary32 addition per
// element), L the levels of the tile tree's binary-counter stack, held in
// registers.  The part's last tile stays in the accumulator (its folded
// value is the lowest entry of the final fold) and needs no level of its
// own, so L levels hold a part of up to 2^L tiles.  Steps past the part end are skipped, so they close no tile and
// add nothing.
template <int BM, int BN, int WM, int WN, int V3_BK, bool F16, int COMB = DG_CARRY, bool FMA0 = false, int L = 1>
__device__ __forceinline__ void v3_body(const GemmArgs& a, int64_t i0, int64_t j0) {
  static_assert(WM * WN == 4, "four waves");
  constexpr bool GEN = COMB != DG_CARRY || FMA0;   // not one carried chain
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / 16, TN = WTN / 16;
  constexpr int ACH = BM * (V3_BK / 8);        // 16-byte chunks per A slab
  constexpr int BCH = V3_BK * (BN / 8);        // 16-byte chunks per B slab
  constexpr int ACH_T = ACH / 256, BCH_T = BCH / 256;
  static_assert(ACH % 256 == 0 && BCH % 256 == 0, "whole chunks per thread");
  constexpr int A_ELEMS = BM * V3_BK, B_ELEMS = V3_BK * BN;   // bf16 per stage
  constexpr int BROW = BN / 8;                 // chunks per B row

  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * (A_ELEMS + B_ELEMS)];
  uint16_t* As0 = smem;
  uint16_t* Bs0 = smem + 2 * A_ELEMS;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int s = blockIdx.z;
  const int64_t k0 = a.cuts[s], k1 = a.cuts[s + 1];
  const int nslab = (int)((k1 - k0 + V3_BK - 1) / V3_BK);

  // A chunk (row, c): LDS chunk row*CPR + (c ^ swz_a<CPR>(row)), CPR = chunks per
  // row (conflict-free fragment reads, as the swizzle's own comment says).
  // B chunk (k, c): LDS chunk k*BROW + (c ^ ((k & 3) << 1)) -- the four rows a
  // transpose read touches land on four different 32-byte bank groups.
  constexpr int CPR = V3_BK / 8;
  static_assert(CPR == 4 || CPR == 8, "BK 32 or 64");
  auto ldsA = [](int row, int c) { return row * CPR + (c ^ swz_a<CPR>(row)); };
  auto ldsB = [](int k, int c) { return k * BROW + (c ^ ((k & 3) << 1)); };

  u32x4 r0a[ACH_T], r0b[BCH_T], r1a[ACH_T], r1b[BCH_T];
  auto gload = [&](int sl, u32x4* ra, u32x4* rb) {
    const int64_t ks = k0 + (int64_t)sl * V3_BK;
#pragma unroll
    for (int t = 0; t < ACH_T; ++t) {
      const int q = tid + 256 * t, row = q / (V3_BK / 8), c = q % (V3_BK / 8);
      const int64_t gi = i0 + row, gk = ks + 8 * c;
      ra[t] = *chunk_or_zero((gi < a.M) && (gk < k1), a.A + gi * a.K + gk);
    }
#pragma unroll
    for (int t = 0; t < BCH_T; ++t) {
      const int q = tid + 256 * t, kr = q / BROW, c = q % BROW;
      const int64_t gk = ks + kr, gn = j0 + 8 * c;
      rb[t] = *chunk_or_zero((gk < k1) && (gn < a.N), a.B + gk * a.N + gn);
    }
  };
  auto lstore = [&](int buf, const u32x4* ra, const u32x4* rb) {
    uint16_t* As = As0 + buf * A_ELEMS;
    uint16_t* Bs = Bs0 + buf * B_ELEMS;
#pragma unroll
    for (int t = 0; t < ACH_T; ++t) {
      const int q = tid + 256 * t;
      *(u32x4*)&As[8 * ldsA(q / (V3_BK / 8), q % (V3_BK / 8))] = ra[t];
    }
#pragma unroll
    for (int t = 0; t < BCH_T; ++t) {
      const int q = tid + 256 * t;
      *(u32x4*)&Bs[8 * ldsB(q / BROW, q % BROW)] = rb[t];
    }
  };

  floatx4 acc[TM][TN];
#pragma unroll
  for (int mi = 0; mi < TM; ++mi)
#pragma unroll
    for (int ni = 0; ni < TN; ++ni) acc[mi][ni] = floatx4{0.f, 0.f, 0.f, 0.f};

  // tile combine state (GEN only): the open tile's accumulator is acc; the
  // chain's running sum or the tree's stack hold the closed tiles
  constexpr int NL = COMB == DG_TREE ? L : COMB == DG_SEQ ? 1 : 0;
  floatx4 stk[NL > 0 ? NL : 1][TM][TN];
  uint32_t count = 0;                                  // tiles closed
  int64_t tile_end = k1;                               // end of the open tile
  if constexpr (GEN) {
    const int64_t len = k1 - k0, tk = a.tile_k;
    const int64_t first = (a.tail_first && len % tk) ? len % tk : tk;
    tile_end = k0 + (first < len ? first : len);
  }
  const floatx4 zero4 = {0.f, 0.f, 0.f, 0.f};
  auto close_tile = [&](bool last) {
    if constexpr (COMB == DG_SEQ) {
      if (count == 0) {
#pragma unroll
        for (int mi = 0; mi < TM; ++mi)
#pragma unroll
          for (int ni = 0; ni < TN; ++ni) stk[0][mi][ni] = acc[mi][ni];
      } else {
#pragma unroll
        for (int mi = 0; mi < TM; ++mi)
#pragma unroll
          for (int ni = 0; ni < TN; ++ni) stk[0][mi][ni] = stk[0][mi][ni] + acc[mi][ni];
      }
    } else if constexpr (COMB == DG_TREE) {
      // binary counter: fold the levels whose bit is set, park at the first clear one
      bool parked = false;
      static_for<0, NL>([&](auto lv) {
        constexpr int LV = decltype(lv)::value;
        if (!parked) {
          if ((count >> LV) & 1u) {
#pragma unroll
            for (int mi = 0; mi < TM; ++mi)
#pragma unroll
              for (int ni = 0; ni < TN; ++ni) acc[mi][ni] = stk[LV][mi][ni] + acc[mi][ni];
          } else {
#pragma unroll
            for (int mi = 0; mi < TM; ++mi)
#pragma unroll
              for (int ni = 0; ni < TN; ++ni) stk[LV][mi][ni] = acc[mi][ni];
            parked = true;
          }
        }
      });
    }
    ++count;
    if (COMB == DG_SEQ || !last) {
#pragma unroll
      for (int mi = 0; mi < TM; ++mi)
#pragma unroll
        for (int ni = 0; ni < TN; ++ni) acc[mi][ni] = zero4;
    }
  };

  auto compute = [&](int buf, int sl) {
    const uint16_t* As = As0 + buf * A_ELEMS;
    const uint16_t* Bs = Bs0 + buf * B_ELEMS;
#pragma unroll
    for (int kk = 0; kk < V3_BK; kk += 32) {
      shortx8 af[TM], bfr[TN];
#pragma unroll
      for (int mi = 0; mi < TM; ++mi) {
        const int row = wm * WTM + 16 * mi + (lane & 15);
        af[mi] = *(const shortx8*)&As[8 * ldsA(row, kk / 8 + (lane >> 4))];
      }
#pragma unroll
      for (int ni = 0; ni < TN; ++ni) {
        const int i = lane & 15, g = lane >> 4;
        const int n = wn * WTN + 16 * ni + 4 * (i & 3);
        const int kr0 = kk + 8 * g + (i >> 2), kr1 = kr0 + 4;
        const shortx4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_s4)(&Bs[8 * ldsB(kr0, n / 8) + (n & 7)]));
        const shortx4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_s4)(&Bs[8 * ldsB(kr1, n / 8) + (n & 7)]));
        bfr[ni] = shortx8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      }
      if constexpr (!GEN) {
#pragma unroll
        for (int mi = 0; mi < TM; ++mi)
#pragma unroll
          for (int ni = 0; ni < TN; ++ni) acc[mi][ni] = mfma16t<F16>(af[mi], bfr[ni], acc[mi][ni]);
      } else {
        const int64_t kpos = k0 + (int64_t)sl * V3_BK + kk;   // this 32-k step (uniform)
        if (kpos < k1) {
#pragma unroll
          for (int mi = 0; mi < TM; ++mi)
#pragma unroll
            for (int ni = 0; ni < TN; ++ni) {
              if constexpr (FMA0) {
                const floatx4 w = mfma16t<F16>(af[mi], bfr[ni], zero4);
                acc[mi][ni] = acc[mi][ni] + w;
              } else {
                acc[mi][ni] = mfma16t<F16>(af[mi], bfr[ni], acc[mi][ni]);
              }
            }
          if constexpr (COMB != DG_CARRY) {
            if (kpos + 32 >= tile_end) {
              close_tile(tile_end >= k1);
              tile_end = tile_end + a.tile_k < k1 ? tile_end + a.tile_k : k1;
            }
          }
        }
      }
    }
  };

  // prologue: slabs 0 and 1 in flight, slab 0 in LDS.  Loads and LDS
  // stores are unconditional (past the part end they read the zero chunk) so
  // that the store of a slab waits only for that slab's loads.
  gload(0, r0a, r0b);
  gload(1, r1a, r1b);
  lstore(0, r0a, r0b);
  __syncthreads();
  for (int sl = 0; sl < nslab; sl += 2) {
    // even slab sl in buffer 0, its successor's registers in set 1
    gload(sl + 2, r0a, r0b);
    compute(0, sl);
    lstore(1, r1a, r1b);
    __syncthreads();
    gload(sl + 3, r1a, r1b);
    if (sl + 1 < nslab) compute(1, sl + 1);
    lstore(0, r0a, r0b);
    __syncthreads();
  }
  // the part's value: the chain's sum, or the tree's stack folded low to high
  if constexpr (COMB == DG_SEQ) {
    if (count) {
#pragma unroll
      for (int mi = 0; mi < TM; ++mi)
#pragma unroll
        for (int ni = 0; ni < TN; ++ni) acc[mi][ni] = stk[0][mi][ni];
    }
  } else if constexpr (COMB == DG_TREE) {
    // acc holds the last tile's folded value, the entry of level ctz(count);
    // the set levels above it meet it in increasing order
    if (count) {
      const int low = __builtin_ctz(count);
      static_for<0, NL>([&](auto lv) {
        constexpr int LV = decltype(lv)::value;
        if (LV > low && ((count >> LV) & 1u)) {
#pragma unroll
          for (int mi = 0; mi < TM; ++mi)
#pragma unroll
            for (int ni = 0; ni < TN; ++ni) acc[mi][ni] = stk[LV][mi][ni] + acc[mi][ni];
        }
      });
    }
  }

  // staging rows of pitch WTN + 4 floats: the four row groups a write
  // instruction covers (rows 4 apart) start 16 banks apart
  constexpr int CSP = WTN + 4;
  float* cs = reinterpret_cast<float*>(smem) + wave * 16 * CSP;
  static_assert(4 * 16 * CSP * 4 <= (int)sizeof(smem), "epilogue staging fits");
#pragma unroll
  for (int mi = 0; mi < TM; ++mi) {
    __syncthreads();
#pragma unroll
    for (int ni = 0; ni < TN; ++ni)
#pragma unroll
      for (int r = 0; r < 4; ++r) cs[(4 * (lane >> 4) + r) * CSP + 16 * ni + (lane & 15)] = acc[mi][ni][r];
    __syncthreads();
#pragma unroll 1
    for (int q = lane; q < 16 * WTN / 4; q += 64) {
      const int rr = q / (WTN / 4), cc = 4 * (q % (WTN / 4));
      const int64_t i = i0 + wm * WTM + 16 * mi + rr, j = j0 + wn * WTN + cc;
      if (i < a.M && j < a.N) finish4(a, s, i, j, *(const float4*)&cs[rr * CSP + cc]);
    }
  }
}

// ---------------------------------------------------------- fp8 tiled
//
// e4m3 x e4m3 with a carried accumulator and fma = 1: the chain of 16-k
// chunks from k = 0, which every fp8 instruction folds alike, issued as the
// block-scaled 16x16x128 (unit scales).  128 x 128 blocks of four 64 x 64
// waves, 128-k slabs (128-byte rows), the v3 pipeline: global loads two
// slabs ahead through two register sets, an LDS double buffer, one barrier
// per slab.
//   * A slab [row][k]: eight 16-byte chunks per row, chunk c at
//     c ^ swz_a<8>(row); a lane's operand is chunk l/16 of its row (bytes
//     0..15) and chunk 4 + l/16 (bytes 16..31): two conflict-free reads;
//   * B slab [k][n]: BN/16 chunks per row, chunk c of row k at c ^ (k & 7),
//     so the 8 rows a transposing read covers sit in 8 different 16-byte
//     slots.  ds_read_b64_tr_b8: lane i of a 16-lane group addresses row
//     i/2, bytes 8(i%2).. of an 8 x 16 byte block and lane j receives
//     column j, byte e from row e; four such reads give a lane its 32 bytes
//     (k = 16(l/16) + 0..7, + 8..15, 64 + 16(l/16) + 0..7, + 8..15);
//   * every 16-byte chunk is wholly inside or outside the part and the
//     matrix (K, N and the part starts are multiples of 16), so a load is a
//     select between a chunk and the zero chunk; a chunk of zero products
//     leaves the accumulator as it is.
typedef __attribute__((address_space(3))) intx2* lds_i2;

__device__ __forceinline__ const u32x4* chunk_or_zero8(bool ok, const uint8_t* p) {
  return ok ? reinterpret_cast<const u32x4*>(p) : &g_zero16[0];
}

template <int BM, int BN>
__device__ __forceinline__ void f8_body(const GemmArgs& a, int64_t i0, int64_t j0) {
  constexpr int WM = 2, WN = 2, WTM = BM / WM, WTN = BN / WN, TM = WTM / 16, TN = WTN / 16;
  constexpr int BK = 128;                        // k per slab (bytes per A row)
  constexpr int CPR = BK / 16, BROW = BN / 16;   // 16-byte chunks per A row, per B row
  constexpr int ACH_T = BM * CPR / 256, BCH_T = BK * BROW / 256;
  static_assert(BM * CPR % 256 == 0 && BK * BROW % 256 == 0, "whole chunks per thread");
  constexpr int A_BYTES = BM * BK, B_BYTES = BK * BN;
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * (A_BYTES + B_BYTES)];
  uint8_t* As0 = smem;
  uint8_t* Bs0 = smem + 2 * A_BYTES;
  const uint8_t* A8 = (const uint8_t*)a.A;
  const uint8_t* B8 = (const uint8_t*)a.B;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int s = blockIdx.z;
  const int64_t k0 = a.cuts[s], k1 = a.cuts[s + 1];
  const int nslab = (int)((k1 - k0 + BK - 1) / BK);
  auto ldsA = [](int row, int c) { return row * CPR + (c ^ swz_a<8>(row)); };
  auto ldsB = [](int k, int c) { return k * BROW + (c ^ (k & 7)); };

  u32x4 r0a[ACH_T], r0b[BCH_T], r1a[ACH_T], r1b[BCH_T];
  auto gload = [&](int sl, u32x4* ra, u32x4* rb) {
    const int64_t ks = k0 + (int64_t)sl * BK;
#pragma unroll
    for (int t = 0; t < ACH_T; ++t) {
      const int q = tid + 256 * t, row = q / CPR, c = q % CPR;
      const int64_t gi = i0 + row, gk = ks + 16 * c;
      ra[t] = *chunk_or_zero8((gi < a.M) && (gk < k1), A8 + gi * a.K + gk);
    }
#pragma unroll
    for (int t = 0; t < BCH_T; ++t) {
      const int q = tid + 256 * t, kr = q / BROW, c = q % BROW;
      const int64_t gk = ks + kr, gn = j0 + 16 * c;
      rb[t] = *chunk_or_zero8((gk < k1) && (gn < a.N), B8 + gk * a.N + gn);
    }
  };
  auto lstore = [&](int buf, const u32x4* ra, const u32x4* rb) {
    uint8_t* As = As0 + buf * A_BYTES;
    uint8_t* Bs = Bs0 + buf * B_BYTES;
#pragma unroll
    for (int t = 0; t < ACH_T; ++t) {
      const int q = tid + 256 * t;
      *(u32x4*)&As[16 * ldsA(q / CPR, q % CPR)] = ra[t];
    }
#pragma unroll
    for (int t = 0; t < BCH_T; ++t) {
      const int q = tid + 256 * t;
      *(u32x4*)&Bs[16 * ldsB(q / BROW, q % BROW)] = rb[t];
    }
  };

  floatx4 acc[TM][TN];
#pragma unroll
  for (int mi = 0; mi < TM; ++mi)
#pragma unroll
    for (int ni = 0; ni < TN; ++ni) acc[mi][ni] = floatx4{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](int buf) {
    const uint8_t* As = As0 + buf * A_BYTES;
    const uint8_t* Bs = Bs0 + buf * B_BYTES;
    const int i = lane & 15, g = lane >> 4;
    intx8 af[TM], bfr[TN];
#pragma unroll
    for (int mi = 0; mi < TM; ++mi) {
      const int row = wm * WTM + 16 * mi + i;
      const u32x4 lo = *(const u32x4*)&As[16 * ldsA(row, g)];
      const u32x4 hi = *(const u32x4*)&As[16 * ldsA(row, 4 + g)];
      af[mi] = intx8{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3], (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
    }
#pragma unroll
    for (int ni = 0; ni < TN; ++ni) {
      const int c = (wn * WTN + 16 * ni) / 16;
      intx2 q[4];
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        const int kr = (h < 2 ? 16 * g + 8 * h : 64 + 16 * g + 8 * (h - 2)) + (i >> 1);
        q[h] = __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_i2)(&Bs[16 * ldsB(kr, c) + 8 * (i & 1)]));
      }
      bfr[ni] = intx8{q[0][0], q[0][1], q[1][0], q[1][1], q[2][0], q[2][1], q[3][0], q[3][1]};
    }
#pragma unroll
    for (int mi = 0; mi < TM; ++mi)
#pragma unroll
      for (int ni = 0; ni < TN; ++ni) acc[mi][ni] = mfma_fp8x128(af[mi], bfr[ni], acc[mi][ni]);
  };

  // prologue: slabs 0 and 1 in flight, slab 0 in LDS (loads past the part
  // end read the zero chunk)
  gload(0, r0a, r0b);
  gload(1, r1a, r1b);
  lstore(0, r0a, r0b);
  __syncthreads();
  for (int sl = 0; sl < nslab; sl += 2) {
    gload(sl + 2, r0a, r0b);
    compute(0);
    lstore(1, r1a, r1b);
    __syncthreads();
    gload(sl + 3, r1a, r1b);
    if (sl + 1 < nslab) compute(1);
    lstore(0, r0a, r0b);
    __syncthreads();
  }

  // epilogue: each wave stages 16-row bands of its tile through LDS (rows of
  // pitch WTN + 4 floats) and finishes four consecutive columns per store
  constexpr int CSP = WTN + 4;
  float* cs = reinterpret_cast<float*>(smem) + wave * 16 * CSP;
  static_assert(4 * 16 * CSP * 4 <= (int)sizeof(smem), "epilogue staging fits");
#pragma unroll
  for (int mi = 0; mi < TM; ++mi) {
    __syncthreads();
#pragma unroll
    for (int ni = 0; ni < TN; ++ni)
#pragma unroll
      for (int r = 0; r < 4; ++r) cs[(4 * (lane >> 4) + r) * CSP + 16 * ni + (lane & 15)] = acc[mi][ni][r];
    __syncthreads();
#pragma unroll 1
    for (int q = lane; q < 16 * WTN / 4; q += 64) {
      const int rr = q / (WTN / 4), cc = 4 * (q % (WTN / 4));
      const int64_t gi = i0 + wm * WTM + 16 * mi + rr, gj = j0 + wn * WTN + cc;
      if (gi < a.M && gj < a.N) finish4(a, s, gi, gj, *(const float4*)&cs[rr * CSP + cc]);
    }
  }
}

template <int BM, int BN>
__global__ __launch_bounds__(256) void gemm_f8(GemmArgs a) {
  const int tiles_n = (int)((a.N + BN - 1) / BN);
  f8_body<BM, BN>(a, (int64_t)(blockIdx.x / tiles_n) * BM, (int64_t)(blockIdx.x % tiles_n) * BN);
}

// Block order (speed only).  order 1: row-major, consecutive workgroups share
// an A panel.  order 2: groups of eight block rows walked column by column.
// order 3: as 2, after giving each XCD (workgroup w runs on XCD w % 8) a
// contiguous range of blocks, so that one XCD's L2 sees neighbouring panels.
__device__ __forceinline__ void grouped_tile(int w, int tiles_m, int tiles_n, int order, int* ty, int* tx) {
  if (order <= 1) {
    *ty = w / tiles_n;
    *tx = w % tiles_n;
    return;
  }
  const int nwg = tiles_m * tiles_n;
  if (order == 3 && nwg % 8 == 0) w = (w % 8) * (nwg / 8) + w / 8;
  constexpr int GROUP = 8;
  const int group = w / (GROUP * tiles_n);
  const int first = group * GROUP;
  const int rows = (tiles_m - first < GROUP) ? tiles_m - first : GROUP;
  const int in_group = w - group * GROUP * tiles_n;
  *ty = first + in_group % rows;
  *tx = in_group / rows;
}

template <int BM, int BN, int WM, int WN, int BK, bool F16>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void gemm_v3(GemmArgs a) {
  const int tiles_m = (int)((a.M + BM - 1) / BM);
  int ty, tx;
  grouped_tile(blockIdx.x, tiles_m, gridDim.x / tiles_m, a.order, &ty, &tx);
  v3_body<BM, BN, WM, WN, BK, F16>(a, (int64_t)ty * BM, (int64_t)tx * BN);
}

// Tile-combine descriptors (chain or tree, or fma = 0) on the v3 pipeline:
// 128 x 128 blocks of four 64 x 64 waves, 32-k slabs, one wave per SIMD.
// The tree's stack takes L x 64 registers per lane at that shape; from four
// levels on the blocks are 128 x 64 (waves of 64 x 32), which halves it.
template <int COMB, int L>
constexpr int tc_bn() { return 64; }
template <int COMB, bool FMA0, int L>
constexpr int tc_bk() { return 32; }
template <int COMB, int L>
constexpr int tc_occ() { return COMB == DG_TREE && L >= 5 ? 1 : 2; }

template <int COMB, bool FMA0, int L, bool F16>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(tc_occ<COMB, L>(), tc_occ<COMB, L>()))) void gemm_tc(GemmArgs a) {
  constexpr int BN = tc_bn<COMB, L>();
  const int tiles_m = (int)((a.M + 127) / 128);
  int ty, tx;
  grouped_tile(blockIdx.x, tiles_m, gridDim.x / tiles_m, a.order, &ty, &tx);
  v3_body<128, BN, 2, 2, tc_bk<COMB, FMA0, L>(), F16, COMB, FMA0, L>(a, (int64_t)ty * 128, (int64_t)tx * BN);
}

template <int BM, int BN, int WM, int WN, int BK, bool F16>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void gemm_v3x2(GemmArgs a) {
  const int tiles_m = (int)((a.M + BM - 1) / BM);
  int ty, tx;
  grouped_tile(blockIdx.x, tiles_m, gridDim.x / tiles_m, a.order, &ty, &tx);
  v3_body<BM, BN, WM, WN, BK, F16>(a, (int64_t)ty * BM, (int64_t)tx * BN);
}

// ------------------------------------------------- ping-pong (eight waves)
//
// Two groups of four waves (one wave of each group per SIMD).  Group g owns
// rows [g BM/2, (g+1) BM/2) of the BM x BN block; each wave a (BM/2) x (BN/4)
// sub-tile.  The groups run the same sequence of phases one phase apart, a
// barrier closing every phase, so that on each SIMD one wave issues MFMAs
// while the other works on LDS:
//   memory phase of slab s: write the group's half of slab s+1 to LDS from
//     registers, read the wave's fragments of slab s;
//   compute phase of slab s: the MFMAs of slab s (its 32-k halves in order),
//     with the loads of the group's half of slab s+3 spread among them (into
//     the register set just written to LDS; two sets alternate).
// Slab s+1's halves are written in phases 2s and 2s+1 and first read in
// phase 2s+2; its buffer last held slab s-1, last read in phase 2s-1.  The
// group that starts late and the group that ends early each take one barrier
// on their own, so every wave takes the same number of barriers.  Slabs past
// the part end are all zero chunks, whose MFMAs leave the accumulators' bits
// unchanged.
//
// Global loads go through buffer resources: a thread's byte offsets inside
// the block are fixed for the launch (a row past M or a column past N gets
// an offset past the resource's end, which reads zero), the slab moves a
// scalar offset, and chunks are checked against the part end only through a
// compare with the elements left.  The host guarantees every offset fits 31
// bits.
// BNC <= BN is the number of columns the block computes; the B slab keeps
// the BN-wide LDS layout and load mapping, and its chunks past BNC are
// neither loaded nor stored.
template <int BM, int BN, int BK, int BNC, bool F16>
__device__ __forceinline__ void pp_body(const GemmArgs& a, int64_t i0, int64_t j0, uint16_t* smem) {
  constexpr int CPR = BK / 8, KK = BK / 32, WTM = BM / 2, WTN = BNC / 4, TM = WTM / 16, TN = WTN / 16;
  constexpr int BROW = BN / 8;
  constexpr int ACH_T = (BM / 2) * CPR / 256, BCH_T = (BK / 2) * BROW / 256;   // per thread
  constexpr int NLOAD = ACH_T + BCH_T, NPAIR = KK * TM;
  static_assert((BM / 2) * CPR % 256 == 0 && (BK / 2) * BROW % 256 == 0 && BROW >= 16, "whole chunks");
  static_assert(CPR == 4 || CPR == 8, "32- or 64-k slabs");
  static_assert(NPAIR >= NLOAD, "at most one load per MFMA group");
  static_assert(BNC <= BN && BNC % 64 == 0, "whole 16-column fragments per wave");
  constexpr int A_ELEMS = BM * BK, B_ELEMS = BK * BN;
  uint16_t* As0 = smem;
  uint16_t* Bs0 = smem + 2 * A_ELEMS;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int grp = wave >> 2, wn = wave & 3, tg = tid & 255;
  const int s = blockIdx.z;
  const int64_t k0 = a.cuts[s], k1 = a.cuts[s + 1];
  const int nslab = (int)((k1 - k0 + BK - 1) / BK);
  // A: chunk c of row r at c ^ swz_a<CPR>(r); B: chunk c of
  // k-row k at c ^ 2 (k % 4) ^ 8 ((k / 8) % 2)
  auto ldsA = [](int row, int c) { return row * CPR + (c ^ swz_a<CPR>(row)); };
  auto ldsB = [](int k, int c) { return k * BROW + (c ^ ((k & 3) << 1) ^ (((k >> 3) & 1) << 3)); };

  constexpr uint32_t OOB = 0x80000000u;
  const int64_t recA = (a.M - i0) * a.K * 2, recB = (a.K - k0) * a.N * 2;
  const __amdgpu_buffer_rsrc_t rA = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a.A + i0 * a.K), (short)0, (int)(recA < 0x7fffffff ? recA : 0x7fffffff), 0x00020000);
  const __amdgpu_buffer_rsrc_t rB = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a.B + k0 * a.N), (short)0, (int)(recB < 0x7fffffff ? recB : 0x7fffffff), 0x00020000);
  // the group's half of a slab: A rows [grp BM/2, +BM/2), B k-rows [grp BK/2, +BK/2)
  uint32_t offA[ACH_T], offB[BCH_T];
  int kcA[ACH_T], kcB[BCH_T];   // the chunk's k within the slab
  int ldA[ACH_T], ldB[BCH_T];   // its LDS chunk
#pragma unroll
  for (int t = 0; t < ACH_T; ++t) {
    const int q = tg + 256 * t, row = grp * (BM / 2) + q / CPR, c = q % CPR;
    offA[t] = (i0 + row < a.M) ? (uint32_t)((row * a.K + 8 * c) * 2) : OOB;
    kcA[t] = 8 * c;
    ldA[t] = ldsA(row, c);
  }
#pragma unroll
  for (int t = 0; t < BCH_T; ++t) {
    const int q = tg + 256 * t, kr = grp * (BK / 2) + q / BROW, c = q % BROW;
    offB[t] = (8 * c < BNC && j0 + 8 * c < a.N) ? (uint32_t)((kr * a.N + j0 + 8 * c) * 2) : OOB;
    kcB[t] = kr;
    ldB[t] = 8 * c < BNC ? ldsB(kr, c) : -1;
  }
  u32x4 ga2[2][ACH_T], gb2[2][BCH_T];
  // load number t of the thread's share of slab sl (A chunks first)
  auto gload1 = [&](int sl, int t, u32x4* ga, u32x4* gb) {
    const int64_t ks = k0 + (int64_t)sl * BK, lim = k1 - ks;
    if (t < ACH_T) {
      const uint32_t off = kcA[t] < lim ? offA[t] : OOB;
      ga[t] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rA, off, (int)(ks * 2), 0));
    } else {
      const int u = t - ACH_T;
      const uint32_t off = kcB[u] < lim ? offB[u] : OOB;
      gb[u] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rB, off, (int)((ks - k0) * a.N * 2), 0));
    }
  };
  auto gload = [&](int sl, u32x4* ga, u32x4* gb) {
#pragma unroll
    for (int t = 0; t < NLOAD; ++t) gload1(sl, t, ga, gb);
  };
  auto lstore = [&](int buf, const u32x4* ga, const u32x4* gb) {
    uint16_t* As = As0 + buf * A_ELEMS;
    uint16_t* Bs = Bs0 + buf * B_ELEMS;
#pragma unroll
    for (int t = 0; t < ACH_T; ++t) *(u32x4*)&As[8 * ldA[t]] = ga[t];
#pragma unroll
    for (int t = 0; t < BCH_T; ++t)
      if (BNC == BN || ldB[t] >= 0) *(u32x4*)&Bs[8 * ldB[t]] = gb[t];
  };

  floatx4 acc[TM][TN];
#pragma unroll
  for (int mi = 0; mi < TM; ++mi)
#pragma unroll
    for (int ni = 0; ni < TN; ++ni) acc[mi][ni] = floatx4{0.f, 0.f, 0.f, 0.f};

  shortx8 af[KK][TM], bf[KK][TN];
  auto rd = [&](int buf) {
    const uint16_t* As = As0 + buf * A_ELEMS;
    const uint16_t* Bs = Bs0 + buf * B_ELEMS;
#pragma unroll
    for (int h = 0; h < KK; ++h) {
#pragma unroll
      for (int ni = 0; ni < TN; ++ni) {
        const int i = lane & 15, g = lane >> 4;
        const int n = wn * WTN + 16 * ni + 4 * (i & 3);
        const int kr0 = 32 * h + 8 * g + (i >> 2), kr1 = kr0 + 4;
        const shortx4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)(&Bs[8 * ldsB(kr0, n / 8) + (n & 7)]));
        const shortx4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)(&Bs[8 * ldsB(kr1, n / 8) + (n & 7)]));
        bf[h][ni] = shortx8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      }
#pragma unroll
      for (int mi = 0; mi < TM; ++mi) {
        const int row = grp * WTM + 16 * mi + (lane & 15);
        af[h][mi] = *(const shortx8*)&As[8 * ldsA(row, 4 * h + (lane >> 4))];
      }
    }
  };
  // MFMAs of pair p: 32-k half p / TM, fragment row p % TM (halves in order)
  auto mm_pair = [&](int p) {
    const int h = p / TM, mi = p % TM;
#pragma unroll
    for (int ni = 0; ni < TN; ++ni) acc[mi][ni] = mfma16t<F16>(af[h][mi], bf[h][ni], acc[mi][ni]);
  };

  // prologue: slab 0 in buffer 0, slabs 1 and 2 in the two register sets
  gload(0, ga2[0], gb2[0]);
  lstore(0, ga2[0], gb2[0]);
  gload(1, ga2[1], gb2[1]);
  gload(2, ga2[0], gb2[0]);
  __syncthreads();
  if (grp == 1) __syncthreads();
  auto step = [&](int sl, u32x4* ga, u32x4* gb) {
    // memory phase: ga/gb hold slab sl+1
    __builtin_amdgcn_sched_barrier(0);
    lstore((sl + 1) & 1, ga, gb);
    rd(sl & 1);
    __syncthreads();
    // compute phase; ga/gb are refilled with slab sl+3
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_setprio(2);
    // load l goes after MFMA group (l + 1) NPAIR / NLOAD - 1
    static_for<0, NPAIR>([&](auto p) {
      mm_pair(p);
      static_for<0, NLOAD>([&](auto l) {
        if constexpr ((l + 1) * NPAIR / NLOAD - 1 == p) {
          __builtin_amdgcn_sched_barrier(0);
          gload1(sl + 3, l, ga, gb);
          __builtin_amdgcn_sched_barrier(0);
        }
      });
    });
    __builtin_amdgcn_s_setprio(0);
    __syncthreads();
  };
  for (int sl = 0; sl < nslab; sl += 2) {
    step(sl, ga2[1], gb2[1]);
    step(sl + 1, ga2[0], gb2[0]);
  }
  if (grp == 0) __syncthreads();

  constexpr int CSP = WTN + 4;
  float* cs = reinterpret_cast<float*>(smem) + wave * 16 * CSP;
  float* bsh = reinterpret_cast<float*>(smem) + 8 * 16 * CSP;
  float* croot = bsh + BNC;   // [group][column]: each group's column roots
  static_assert((8 * 16 * CSP + 3 * BNC) * 4 <= 2 * (A_ELEMS + B_ELEMS) * 2, "epilogue staging fits");
  __syncthreads();
  stage_bias(a, j0, BNC, bsh);
  __syncthreads();
  // a 256-row block is one run of the column sums: each group folds its 128
  // rows, and the two roots meet (group 0's rows first)
  const bool tree = BM == 256 && a.colsum_part != nullptr;
  wave_epilogue<TM, TN>(a, s, i0 + grp * WTM, j0 + wn * WTN, cs, bsh + wn * WTN, acc,
                        tree ? croot + grp * BNC + wn * WTN : nullptr);
  if (tree) {
    __syncthreads();
    for (int c = tid; c < BNC; c += 512)
      if (j0 + c < a.N) a.colsum_part[(i0 / 256) * a.N + j0 + c] = croot[c] + croot[BNC + c];
  }
}

// ------------------------------------- ping-pong with direct-to-LDS loads
//
// The same eight-wave schedule and LDS layouts as pp_body for 256 x BNC
// blocks and 32-k slabs, but the loads go from memory straight into LDS
// (buffer_load ... lds: lane l's 16 bytes land at the instruction's LDS base
// + 16 l), so no staging registers and no LDS write instructions remain:
// VGPR->LDS writes run at under 100 B/clk per CU on MI355X against ~230 for
// reads, and they were the largest single cost of the register-staged
// schedule.  Each lane fetches the chunk that belongs at its LDS slot under
// the swizzle (the XOR maps are involutions), so the layouts are unchanged.
//
// A ring of four slots (one slab each, in four separate LDS arrays so that
// the compiler tells them apart and waits only for the slot it reads): the
// loads of slab s+3 are issued during the compute phase of slab s into the
// slot that slab s-1 left.  A group's loads are complete once its own
// outstanding count allows it, and visible to the other group after the
// next barrier:
//   group 0 ends each compute phase with at most two slabs of its loads in
//   flight (s+2, s+3), group 1 ends each memory phase with at most one
//   (s+2), so slab s+1 is in LDS, from both groups, at the barrier that
//   precedes group 0's memory phase of s+1.
constexpr int PPD_SLOT = 256 * 32 + 32 * 256;   // bf16 elements per slot
__shared__ __attribute__((aligned(1024))) uint16_t ppd_s0[PPD_SLOT];
__shared__ __attribute__((aligned(1024))) uint16_t ppd_s1[PPD_SLOT];
__shared__ __attribute__((aligned(1024))) uint16_t ppd_s2[PPD_SLOT];
__shared__ __attribute__((aligned(1024))) uint16_t ppd_s3[PPD_SLOT];

template <int S>
__device__ __forceinline__ uint16_t* ppd_slot() {
  if constexpr (S == 0) return ppd_s0;
  else if constexpr (S == 1) return ppd_s1;
  else if constexpr (S == 2) return ppd_s2;
  else return ppd_s3;
}

typedef __attribute__((address_space(3))) void* lds_void;


// Workgroup barrier without the memory fence of __syncthreads: the fence
// would make every wave wait for all of its direct-to-LDS loads.  The loads
// a phase needs are waited for explicitly (vmcnt) before it.
__device__ __forceinline__ void barrier_nofence() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

template <int BNC>
__device__ __forceinline__ void ppd_body(const GemmArgs& a, int64_t i0, int64_t j0) {
  constexpr int BM = 256, BN = 256, BK = 32, CPR = 4, WTM = 128, WTN = BNC / 4, TM = 8, TN = WTN / 16;
  constexpr int A_ELEMS = BM * BK;
  constexpr int NL = 4;                     // loads per thread per slab: 2 of A, 2 of B
  constexpr int NPAIR = TM;                 // MFMA groups per compute phase
  static_assert(BNC <= BN && BNC % 64 == 0, "whole 16-column fragments per wave");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int grp = wave >> 2, wn = wave & 3;
  const int s = blockIdx.z;
  const int64_t k0 = a.cuts[s], k1 = a.cuts[s + 1];
  const int nslab = (int)((k1 - k0 + BK - 1) / BK);
  auto ldsA = [](int row, int c) { return row * CPR + (c ^ swz_a<CPR>(row)); };
  auto ldsB = [](int k, int c) { return k * (BN / 8) + (c ^ ((k & 3) << 1) ^ (((k >> 3) & 1) << 3)); };

  constexpr uint32_t OOB = 0x80000000u;
  const int64_t recA = (a.M - i0) * a.K * 2, recB = (a.K - k0) * a.N * 2;
  const __amdgpu_buffer_rsrc_t rA = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a.A + i0 * a.K), (short)0, (int)(recA < 0x7fffffff ? recA : 0x7fffffff), 0x00020000);
  const __amdgpu_buffer_rsrc_t rB = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a.B + k0 * a.N), (short)0, (int)(recB < 0x7fffffff ? recB : 0x7fffffff), 0x00020000);
  // Load i of the thread's share, i = 0, 1: A rows grp*128 + (wn*2+i)*16 +
  // lane/4 (physical chunk lane%4), then B k-rows grp*16 + (wn*2+i)*2 +
  // lane/32 (physical chunk lane%32).  Each instruction fills 1 KB of LDS.
  uint32_t offA[2], offB[2];
  int kcA[2], kcB[2], dA[2], dB[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int r = grp * 128 + (wn * 2 + i) * 16 + lane / 4, pc = lane & 3;
    const int c = pc ^ swz_a<CPR>(r);
    offA[i] = (i0 + r < a.M) ? (uint32_t)((r * a.K + 8 * c) * 2) : OOB;
    kcA[i] = 8 * c;
    dA[i] = (grp * 128 + (wn * 2 + i) * 16) * BK;           // element offset of the 1 KB run
    const int kr = grp * 16 + (wn * 2 + i) * 2 + lane / 32, pb = lane & 31;
    const int cb = pb ^ ((kr & 3) << 1) ^ (((kr >> 3) & 1) << 3);
    offB[i] = (8 * cb < BNC && j0 + 8 * cb < a.N) ? (uint32_t)((kr * a.N + j0 + 8 * cb) * 2) : OOB;
    kcB[i] = kr;
    dB[i] = A_ELEMS + (grp * 16 + (wn * 2 + i) * 2) * BN;
  }
  // load l (0, 1: A; 2, 3: B) of slab sl into slot S
  auto dma1 = [&](auto S, int sl, int l) {
    uint16_t* base = ppd_slot<decltype(S)::value>();
    const int64_t ks = k0 + (int64_t)sl * BK, lim = k1 - ks;
    if (l < 2) {
      const uint32_t off = kcA[l] < lim ? offA[l] : OOB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rA, (lds_void)(base + dA[l]), 16, off, (int)(ks * 2), 0, 0);
    } else {
      const int i = l - 2;
      const uint32_t off = kcB[i] < lim ? offB[i] : OOB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rB, (lds_void)(base + dB[i]), 16, off, (int)((ks - k0) * a.N * 2), 0, 0);
    }
  };

  floatx4 acc[TM][TN];
#pragma unroll
  for (int mi = 0; mi < TM; ++mi)
#pragma unroll
    for (int ni = 0; ni < TN; ++ni) acc[mi][ni] = floatx4{0.f, 0.f, 0.f, 0.f};
  shortx8 af[TM], bf[TN];
  auto rd = [&](auto S) {
    const uint16_t* As = ppd_slot<decltype(S)::value>();
    const uint16_t* Bs = As + A_ELEMS;
#pragma unroll
    for (int ni = 0; ni < TN; ++ni) {
      const int i = lane & 15, g = lane >> 4;
      const int n = wn * WTN + 16 * ni + 4 * (i & 3);
      const int kr0 = 8 * g + (i >> 2), kr1 = kr0 + 4;
      const shortx4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)(&Bs[8 * ldsB(kr0, n / 8) + (n & 7)]));
      const shortx4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)(&Bs[8 * ldsB(kr1, n / 8) + (n & 7)]));
      bf[ni] = shortx8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    }
#pragma unroll
    for (int mi = 0; mi < TM; ++mi) {
      const int row = grp * WTM + 16 * mi + (lane & 15);
      af[mi] = *(const shortx8*)&As[8 * ldsA(row, lane >> 4)];
    }
  };

  // prologue: slabs 0, 1, 2 into slots 0, 1, 2; slab 0 complete everywhere
  static_for<0, NL>([&](auto l) { dma1(std::integral_constant<int, 0>{}, 0, l); });
  static_for<0, NL>([&](auto l) { dma1(std::integral_constant<int, 1>{}, 1, l); });
  static_for<0, NL>([&](auto l) { dma1(std::integral_constant<int, 2>{}, 2, l); });
  __builtin_amdgcn_s_waitcnt(vmcnt_only(2 * NL));
  barrier_nofence();
  if (grp == 1) barrier_nofence();
  auto step = [&](auto S, int sl) {
    constexpr int SL = decltype(S)::value;
    // memory phase: fragments of slab sl
    __builtin_amdgcn_sched_barrier(0);
    rd(S);
    if (grp == 1) __builtin_amdgcn_s_waitcnt(vmcnt_only(NL));   // slab sl+1 landed
    barrier_nofence();
    // compute phase: the MFMAs of slab sl, the loads of slab sl+3 spread among them
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_setprio(2);
    static_for<0, NPAIR>([&](auto p) {
#pragma unroll
      for (int ni = 0; ni < TN; ++ni) acc[p][ni] = mfma16(af[p], bf[ni], acc[p][ni]);
      static_for<0, NL>([&](auto l) {
        if constexpr ((l + 1) * NPAIR / NL - 1 == p) {
          __builtin_amdgcn_sched_barrier(0);
          dma1(std::integral_constant<int, (SL + 3) % 4>{}, sl + 3, l);
          __builtin_amdgcn_sched_barrier(0);
        }
      });
    });
    __builtin_amdgcn_s_setprio(0);
    if (grp == 0) __builtin_amdgcn_s_waitcnt(vmcnt_only(2 * NL));   // slab sl+1 landed
    barrier_nofence();
  };
  for (int sl = 0; sl < nslab; sl += 4) {
    step(std::integral_constant<int, 0>{}, sl);
    step(std::integral_constant<int, 1>{}, sl + 1);
    step(std::integral_constant<int, 2>{}, sl + 2);
    step(std::integral_constant<int, 3>{}, sl + 3);
  }
  if (grp == 0) barrier_nofence();
  // loads of slabs past the end (zeros) may still be landing in the slots
  __builtin_amdgcn_s_waitcnt(vmcnt_only(0));
  __syncthreads();

  // epilogue: wave w stages through slot w % 4, at (w / 4) * 16 rows of pitch
  // CSP; the bias sits in slot 0 after its two staging areas
  constexpr int CSP = WTN + 4;
  static_assert((2 * 16 * CSP + BNC) * 4 <= PPD_SLOT * 2, "epilogue staging fits");
  uint16_t* sb = (wave & 3) == 0 ? ppd_s0 : (wave & 3) == 1 ? ppd_s1 : (wave & 3) == 2 ? ppd_s2 : ppd_s3;
  float* cs = reinterpret_cast<float*>(sb) + (wave >> 2) * 16 * CSP;
  float* bsh = reinterpret_cast<float*>(ppd_s0) + 2 * 16 * CSP;
  stage_bias(a, j0, BNC, bsh);
  __syncthreads();
  wave_epilogue<TM, TN>(a, s, i0 + grp * WTM, j0 + wn * WTN, cs, bsh + wn * WTN, acc);
}

__global__ __launch_bounds__(512) void gemm_ppd(GemmArgs a) {
  const int tiles_m = (int)((a.M + 255) / 256);
  int ty, tx;
  grouped_tile(blockIdx.x, tiles_m, gridDim.x / tiles_m, a.order, &ty, &tx);
  ppd_body<256>(a, (int64_t)ty * 256, (int64_t)tx * 256);
}

__global__ __launch_bounds__(512) void gemm_ppd_mixed(GemmArgs a) {
  const int tiles_m = (int)((a.M + 255) / 256);
  const int tn1 = (int)(a.n_split / 256), nb1 = tiles_m * tn1;
  int ty, tx;
  if ((int)blockIdx.x < nb1) {
    grouped_tile(blockIdx.x, tiles_m, tn1, a.order, &ty, &tx);
    ppd_body<256>(a, (int64_t)ty * 256, (int64_t)tx * 256);
  } else {
    const int tn2 = (int)((a.N - a.n_split + 191) / 192);
    grouped_tile(blockIdx.x - nb1, tiles_m, tn2, a.order, &ty, &tx);
    ppd_body<192>(a, (int64_t)ty * 256, a.n_split + (int64_t)tx * 192);
  }
}

template <int BM, int BN, int BK, bool F16>
__global__ __launch_bounds__(512) void gemm_pp(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * (BM * BK + BK * BN)];
  const int tiles_m = (int)((a.M + BM - 1) / BM);
  int ty, tx;
  grouped_tile(blockIdx.x, tiles_m, gridDim.x / tiles_m, a.order, &ty, &tx);
  pp_body<BM, BN, BK, BN, F16>(a, (int64_t)ty * BM, (int64_t)tx * BN, smem);
}

// Two column widths in one launch: columns [0, n_split) in 256 x 256 blocks
// (the first workgroups), the rest in 256 x 192 blocks.  With one block per
// CU, a width mix can make the work a whole number of rounds over the chip
// where 256-wide blocks alone leave the last round partly idle (2048 x 14336:
// 448 blocks of 256 x 256 take two rounds on 256 CUs; 256 blocks of
// 256 x 256 and 256 of 256 x 192 take 1.75 rounds of work).
template <int BK, bool F16>
__global__ __launch_bounds__(512) void gemm_pp_mixed(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * (256 * BK + BK * 256)];
  const int tiles_m = (int)((a.M + 255) / 256);
  const int tn1 = (int)(a.n_split / 256), nb1 = tiles_m * tn1;
  int ty, tx;
  if ((int)blockIdx.x < nb1) {
    grouped_tile(blockIdx.x, tiles_m, tn1, a.order, &ty, &tx);
    pp_body<256, 256, BK, 256, F16>(a, (int64_t)ty * 256, (int64_t)tx * 256, smem);
  } else {
    const int tn2 = (int)((a.N - a.n_split + 191) / 192);
    grouped_tile(blockIdx.x - nb1, tiles_m, tn2, a.order, &ty, &tx);
    pp_body<256, 256, BK, 192, F16>(a, (int64_t)ty * 256, a.n_split + (int64_t)tx * 192, smem);
  }
}

// ------------------------------------ four waves, 128-row wave sub-tiles
//
// One wave per SIMD, each owning a 128 x (BNC/2) sub-tile of the 256 x BNC
// block with its accumulators (up to 256 registers) in the accumulation
// register file, tied to the MFMAs through inline assembly.  Against the
// eight-wave ping-pong this reads a third fewer fragment bytes from LDS per
// MFMA (each A fragment is read by two waves, not four).  The slabs move by
// direct-to-LDS loads (lane l's 16 bytes land at the instruction's LDS base
// + 16 l; each lane fetches the chunk that belongs at its position under the
// swizzle) into a ring of NS slots, D = NS - 1 slabs ahead: per 32-k slab
// each wave issues eight such loads and no LDS write (a register-staged
// version issued eight global loads and eight LDS writes and ran ~6 %
// slower).  Iteration s: MFMAs of slab s, fragments of slab s+1 read from
// slot (s+1) % NS, loads of slab s+D into slot (s+D) % NS (whose slab s-1 was
// consumed in iteration s-1), then a wait until the wave's loads of slab s+2
// have landed, and one barrier.
constexpr int W4D_SLOT = 256 * 32 + 32 * 256;   // bf16 elements per slot
__shared__ __attribute__((aligned(1024))) uint16_t w4d_s0[W4D_SLOT];
__shared__ __attribute__((aligned(1024))) uint16_t w4d_s1[W4D_SLOT];
__shared__ __attribute__((aligned(1024))) uint16_t w4d_s2[W4D_SLOT];
__shared__ __attribute__((aligned(1024))) uint16_t w4d_s3[W4D_SLOT];

template <int S>
__device__ __forceinline__ uint16_t* w4d_slot() {
  if constexpr (S == 0) return w4d_s0;
  else if constexpr (S == 1) return w4d_s1;
  else if constexpr (S == 2) return w4d_s2;
  else return w4d_s3;
}

template <int BNC>
__device__ __forceinline__ void w4d_body(const GemmArgs& a, int64_t i0, int64_t j0) {
  constexpr int NS = 4;   // four separate LDS arrays, so that the compiler tells the slots apart
  constexpr int BM = 256, BN = 256, BK = 32, CPR = BK / 8, BROW = BN / 8, D = NS - 1;
  constexpr int WTM = 128, WTN = BNC / 2, TM = WTM / 16, TN = WTN / 16;
  constexpr int A_ELEMS = BM * BK, B_ELEMS = BK * BN, SLOT = A_ELEMS + B_ELEMS;
  constexpr int NIA = A_ELEMS * 2 / 1024 / 4, NIB = B_ELEMS * 2 / 1024 / 4, NI = NIA + NIB;   // per wave
  static_assert(BNC <= BN && BNC % 32 == 0 && TN <= TM && D >= 2 && NI == TM, "one load per MFMA group");
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int s = blockIdx.z;
  const int64_t k0 = a.cuts[s], k1 = a.cuts[s + 1];
  const int nslab = (int)((k1 - k0 + BK - 1) / BK);
  auto ldsA = [](int row, int c) { return row * CPR + (c ^ swz_a<CPR>(row)); };
  auto ldsB = [](int k, int c) { return k * BROW + (c ^ ((k & 3) << 1) ^ (((k >> 3) & 1) << 3)); };

  // load t of the wave: A run r = NIA wave + t (16 rows of 64 bytes), B run
  // r = NIB wave + (t - NIA) (2 k-rows of 512 bytes)
  constexpr uint32_t OOB = 0x80000000u;
  uint32_t off[NI];
  int kc[NI];
#pragma unroll
  for (int t = 0; t < NIA; ++t) {
    const int row = (NIA * wave + t) * 16 + lane / 4, pc = lane % 4;
    const int c = pc ^ swz_a<CPR>(row);
    off[t] = (i0 + row < a.M) ? (uint32_t)((row * a.K + 8 * c) * 2) : OOB;
    kc[t] = 8 * c;
  }
#pragma unroll
  for (int u = 0; u < NIB; ++u) {
    const int kr = (NIB * wave + u) * 2 + lane / 32, pc = lane % 32;
    const int c = pc ^ ((kr & 3) << 1) ^ (((kr >> 3) & 1) << 3);
    off[NIA + u] = (8 * c < BNC && j0 + 8 * c < a.N) ? (uint32_t)((kr * a.N + j0 + 8 * c) * 2) : OOB;
    kc[NIA + u] = kr;
  }
  const int64_t recA = (a.M - i0) * a.K * 2, recB = (a.K - k0) * a.N * 2;
  const __amdgpu_buffer_rsrc_t rA = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a.A + i0 * a.K), (short)0, (int)(recA < 0x7fffffff ? recA : 0x7fffffff), 0x00020000);
  const __amdgpu_buffer_rsrc_t rB = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a.B + k0 * a.N), (short)0, (int)(recB < 0x7fffffff ? recB : 0x7fffffff), 0x00020000);
  // load t of slab sl into slot `slot`; past the part end: zeros, slab offset 0
  auto dma1 = [&](int sl_in, auto SL, auto T) {
    constexpr int t = decltype(T)::value;
    const bool past = sl_in >= nslab;
    const int sl = past ? 0 : sl_in;
    const int64_t ks = k0 + (int64_t)sl * BK, lim = past ? 0 : k1 - ks;
    uint16_t* base = w4d_slot<decltype(SL)::value>();
    if constexpr (t < NIA)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rA, (lds_void)(base + (NIA * wave + t) * 512), 16,
                                               kc[t] < lim ? off[t] : OOB, (int)(ks * 2), 0, 0);
    else
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rB, (lds_void)(base + A_ELEMS + (NIB * wave + t - NIA) * 512), 16,
                                               kc[t] < lim ? off[t] : OOB, (int)((ks - k0) * a.N * 2), 0, 0);
  };

  floatx4 acc[TM][TN];
#pragma unroll
  for (int mi = 0; mi < TM; ++mi)
#pragma unroll
    for (int ni = 0; ni < TN; ++ni) acc[mi][ni] = floatx4{0.f, 0.f, 0.f, 0.f};
  shortx8 fa[2][TM], fb[2][TN];
  auto rdA = [&](auto SL, int mi, shortx8& f) {
    const int row = wm * WTM + 16 * mi + (lane & 15);
    f = *(const shortx8*)&w4d_slot<decltype(SL)::value>()[8 * ldsA(row, lane >> 4)];
  };
  auto rdB = [&](auto SL, int ni, shortx8& f) {
    const uint16_t* Bs = w4d_slot<decltype(SL)::value>() + A_ELEMS;
    const int i = lane & 15, gq = lane >> 4;
    const int n = wn * WTN + 16 * ni + 4 * (i & 3);
    const int kr0 = 8 * gq + (i >> 2), kr1 = kr0 + 4;
    const shortx4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)(&Bs[8 * ldsB(kr0, n / 8) + (n & 7)]));
    const shortx4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)(&Bs[8 * ldsB(kr1, n / 8) + (n & 7)]));
    f = shortx8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  };

  // prologue: slabs 0 .. D-1 issued, 0 and 1 landed (all waves), slab 0's
  // fragments read
  static_for<0, D>([&](auto x) { static_for<0, NI>([&](auto t) { dma1(x, x, t); }); });
  __builtin_amdgcn_s_waitcnt(vmcnt_only((D - 2) * NI));
  barrier_nofence();
  constexpr std::integral_constant<int, 0> S0{};
#pragma unroll
  for (int mi = 0; mi < TM; ++mi) rdA(S0, mi, fa[0][mi]);
#pragma unroll
  for (int ni = 0; ni < TN; ++ni) rdB(S0, ni, fb[0][ni]);
  lds_wait();
  barrier_nofence();

  auto step = [&](int sl, auto X) {
    constexpr int x = decltype(X)::value, cur = x & 1, nxt = cur ^ 1;
    constexpr std::integral_constant<int, (x + 1) % NS> rslot{};
    constexpr std::integral_constant<int, (x + D) % NS> wslot{};
    __builtin_amdgcn_sched_barrier(0);
    static_for<0, TM>([&](auto mi) {
#pragma unroll
      for (int ni = 0; ni < TN; ++ni) mfma16_tied(acc[mi][ni], fa[cur][mi], fb[cur][ni]);
      __builtin_amdgcn_sched_barrier(0);
      rdA(rslot, mi, fa[nxt][mi]);
      if constexpr (mi < TN) rdB(rslot, mi, fb[nxt][mi]);
      dma1(sl + D, wslot, mi);
      __builtin_amdgcn_sched_barrier(0);
    });
    lds_wait();
    __builtin_amdgcn_s_waitcnt(vmcnt_only((D - 2) * NI));   // the wave's loads of slab sl+2 landed
    barrier_nofence();
  };
  for (int sl = 0; sl < nslab; sl += NS)
    static_for<0, NS>([&](auto x) { step(sl + x, x); });
  mfma_drain();
  __builtin_amdgcn_s_waitcnt(vmcnt_only(0));   // nothing lands in the staging area later
  barrier_nofence();

  // epilogue: wave w stages through slot w; the bias sits in slot 0 after
  // wave 0's area
  constexpr int CSP = WTN + 4;
  static_assert((16 * CSP + BNC) * 4 <= SLOT * 2, "epilogue staging fits");
  uint16_t* sb = wave == 0 ? w4d_s0 : wave == 1 ? w4d_s1 : wave == 2 ? w4d_s2 : w4d_s3;
  float* cs = reinterpret_cast<float*>(sb);
  float* bsh = reinterpret_cast<float*>(w4d_s0) + 16 * CSP;
  stage_bias(a, j0, BNC, bsh);
  __syncthreads();
  wave_epilogue<TM, TN>(a, s, i0 + wm * WTM, j0 + wn * WTN, cs, bsh + wn * WTN, acc);
}

// e4m3 x e4m3 (carried accumulator, fma = 1) on 256 x 256 blocks of four
// 128 x 128 waves, or 256 x 128 blocks of four 128 x 64 waves (two blocks
// per CU): the w4d pipeline above with bytes for bf16 elements.
// The slab is 64 k, so A rows are 64 bytes (the bf16 slab's layout and
// swizzle) and the instruction is the block-scaled 32x32x64 (unit scales),
// whose K is the slab: lane l's bytes 0..15 are k = 16(l/32) + e, bytes
// 16..31 k = 32 + 16(l/32) + e, row (A) or column (B) l % 32; its 16
// results are rows 8(r/4) + 4(l/32) + r%4 of column l % 32.  B rows are 256
// bytes, chunk c of row k at c ^ (k & 7) ^ 8 (c & 1), read through
// ds_read_b64_tr_b8 as in the 128 x 128 kernel: a read pass serves two
// 16-lane groups, on neighbouring chunks of the same 8 rows, and the odd
// chunk's rows sit in the other half of the 256-byte row (all 64 banks).
// Per slab each wave issues four A and four B direct-to-LDS loads (16 rows
// of A or 4 rows of B per 1 KB run) and 16 MFMAs; the accumulators (256
// floats) live in the accumulation registers.  The ring has four slots
// and runs four slabs ahead: slab s's slot is free once its fragments are
// in registers (the barrier ending step s - 1), so step s loads slab s + 4
// into it, and a load has two to three steps to land (fp8 spends half the
// bf16 kernel's MFMA time on a slab of the same bytes).  Each slot is two
// LDS arrays (A, B): the compiler
// keeps a fragment read apart from the direct-to-LDS loads still in flight
// only when they touch different arrays (it tracks up to eight), and with
// one array per slot it made every B-fragment read wait for all of them.
__shared__ __attribute__((aligned(1024))) uint8_t f8w_a0[16384];
__shared__ __attribute__((aligned(1024))) uint8_t f8w_a1[16384];
__shared__ __attribute__((aligned(1024))) uint8_t f8w_a2[16384];
__shared__ __attribute__((aligned(1024))) uint8_t f8w_a3[16384];
__shared__ __attribute__((aligned(1024))) uint8_t f8w_b0[16384];
__shared__ __attribute__((aligned(1024))) uint8_t f8w_b1[16384];
__shared__ __attribute__((aligned(1024))) uint8_t f8w_b2[16384];
__shared__ __attribute__((aligned(1024))) uint8_t f8w_b3[16384];
template <int S>
__device__ __forceinline__ uint8_t* f8w_aslot() {
  if constexpr (S == 0) return f8w_a0;
  else if constexpr (S == 1) return f8w_a1;
  else if constexpr (S == 2) return f8w_a2;
  else return f8w_a3;
}
// The 256 x 128 blocks' B slots (64 x 128 bytes): a block then takes
// 72 KB of LDS and registers for two waves per SIMD, so two blocks share a
// CU and one's prologue and epilogue run beside the other's main loop.
__shared__ __attribute__((aligned(1024))) uint8_t f8n_b0[8192];
__shared__ __attribute__((aligned(1024))) uint8_t f8n_b1[8192];
__shared__ __attribute__((aligned(1024))) uint8_t f8n_b2[8192];
template <int BN, int S>
__device__ __forceinline__ uint8_t* f8w_bslot() {
  if constexpr (BN == 128) {
    if constexpr (S == 0) return f8n_b0;
    else if constexpr (S == 1) return f8n_b1;
    else return f8n_b2;
  } else {
    if constexpr (S == 0) return f8w_b0;
    else if constexpr (S == 1) return f8w_b1;
    else if constexpr (S == 2) return f8w_b2;
    else return f8w_b3;
  }
}

// BN 256: four slots; BN 128 (waves of 128 x 64): three slots.  EB is the
// operand's bytes: 1 (e4m3, 64-k slabs, the block-scaled 32x32x64) or 2
// (bf16, 32-k slabs of the same bytes, two 32x32x16 bf16 instructions per
// slab in k order -- the bf16 chain of 8-k chunks; 256 x 128 blocks only).
template <int BN, int EB = 1>
__device__ __forceinline__ void f8w_body(const GemmArgs& a, int64_t i0, int64_t j0) {
  constexpr int NS = BN == 256 ? 4 : 3, D = NS;
  constexpr int EPC = 16 / EB;                                  // elements per 16-byte chunk
  constexpr int BM = 256, BK = 64 / EB, CPR = 4, BROW = BN * EB / 16;
  constexpr int WTM = 128, WTN = BN / 2, TM = WTM / 32, TN = WTN / 32;
  constexpr int A_BYTES = BM * BK * EB, B_BYTES = BK * BN * EB;
  static_assert(EB == 1 || BN == 128, "bf16: 256 x 128 blocks");
  constexpr int NIA = A_BYTES / 1024 / 4, NIB = B_BYTES / 1024 / 4, NI = NIA + NIB;   // per wave
  constexpr int BRUN = 1024 / (16 * BROW);                                            // B rows per 1 KB run
  static_assert((BN == 256 || BN == 128) && TN <= TM && A_BYTES == 16384, "block shapes");
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int s = blockIdx.z;
  const int64_t k0 = a.cuts[s], k1 = a.cuts[s + 1];
  const int nslab = (int)((k1 - k0 + BK - 1) / BK);
  auto ldsA = [](int row, int c) { return row * CPR + (c ^ swz_a<CPR>(row)); };
  // e4m3, 128-byte B rows: two rows span the 64 banks, so c ^ (k & 7)
  // already spreads a transposing read's 8 rows and two groups over them.
  // bf16 (256-byte rows, 4-row transposing reads of 32 bytes per 16-lane
  // group): c ^ 4 (k & 3) gives the 4 rows of both groups of a pass 16
  // different chunks.
  auto ldsB = [](int k, int c) {
    if constexpr (EB == 2) return k * BROW + (c ^ ((k & 3) << 2));
    else return k * BROW + (c ^ (k & 7) ^ (BROW == 16 ? (c & 1) << 3 : 0));
  };

  // load t of the wave: A run r = NIA wave + t (rows 16r..), B run
  // r = NIB wave + (t - NIA) (k rows BRUN r..); each lane fetches the chunk
  // that belongs at its LDS position under the swizzle
  constexpr uint32_t OOB = 0x80000000u;
  uint32_t off[NI];
  int kc[NI];
#pragma unroll
  for (int t = 0; t < NIA; ++t) {
    const int row = (NIA * wave + t) * 16 + lane / 4, pc = lane % 4;
    const int c = pc ^ swz_a<CPR>(row);
    off[t] = (i0 + row < a.M) ? (uint32_t)(row * a.K * EB + 16 * c) : OOB;
    kc[t] = EPC * c;
  }
#pragma unroll
  for (int u = 0; u < NIB; ++u) {
    const int kr = (NIB * wave + u) * BRUN + lane / BROW, pc = lane % BROW;
    // the chunk stored at position pc
    const int c = EB == 2 ? pc ^ ((kr & 3) << 2) : pc ^ (kr & 7) ^ (BROW == 16 ? ((pc ^ kr) & 1) << 3 : 0);
    off[NIA + u] = (j0 + EPC * c < a.N) ? (uint32_t)((kr * a.N + j0 + EPC * c) * EB) : OOB;
    kc[NIA + u] = kr;
  }
  const uint8_t* A8 = (const uint8_t*)a.A;
  const uint8_t* B8 = (const uint8_t*)a.B;
  const int64_t recA = (a.M - i0) * a.K * EB, recB = (a.K - k0) * a.N * EB;   // below 2^31 (host check)
  const __amdgpu_buffer_rsrc_t rA = __builtin_amdgcn_make_buffer_rsrc((void*)(A8 + i0 * a.K * EB), (short)0,
                                                                      (int)recA, 0x00020000);
  const __amdgpu_buffer_rsrc_t rB = __builtin_amdgcn_make_buffer_rsrc((void*)(B8 + k0 * a.N * EB), (short)0,
                                                                      (int)recB, 0x00020000);
  auto dma1 = [&](int sl_in, auto SL, auto T) {
    constexpr int t = decltype(T)::value;
    const bool past = sl_in >= nslab;
    const int sl = past ? 0 : sl_in;
    const int64_t ks = k0 + (int64_t)sl * BK, lim = past ? 0 : k1 - ks;
    constexpr int sl_ = decltype(SL)::value;
    if constexpr (t < NIA)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rA, (lds_void)(f8w_aslot<sl_>() + (NIA * wave + t) * 1024), 16,
                                               kc[t] < lim ? off[t] : OOB, (int)(ks * EB), 0, 0);
    else
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rB, (lds_void)(f8w_bslot<BN, sl_>() + (NIB * wave + t - NIA) * 1024), 16,
                                               kc[t] < lim ? off[t] : OOB, (int)((ks - k0) * a.N * EB), 0, 0);
  };

  floatx16 acc[TM][TN];
#pragma unroll
  for (int mi = 0; mi < TM; ++mi)
#pragma unroll
    for (int ni = 0; ni < TN; ++ni)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mi][ni][r] = 0.f;
  // bf16 keeps one set of A fragments (a row's next fragment is read once
  // that row's MFMAs are issued), so that the block fits two waves per SIMD
  constexpr int FA = EB == 2 ? 1 : 2;
  intx8 fa[FA][TM], fb[2][TN];
  auto rdA = [&](auto SL, int mi, intx8& f) {
    const uint8_t* As = f8w_aslot<decltype(SL)::value>();
    const int row = wm * WTM + 32 * mi + (lane & 31), h = lane >> 5;
    const u32x4 lo = *(const u32x4*)&As[16 * ldsA(row, h)];
    const u32x4 hi = *(const u32x4*)&As[16 * ldsA(row, 2 + h)];
    f = intx8{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3], (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
  };
  auto rdB = [&](auto SL, int ni, intx8& f) {
    const uint8_t* Bs = f8w_bslot<BN, decltype(SL)::value>();
    const int q = lane >> 4, i = lane & 15, h = q >> 1;
    intx2 v[4];
    if constexpr (EB == 1) {
      const int c = (wn * WTN + 32 * ni + 16 * (q & 1)) / 16;
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const int kr = (p < 2 ? 16 * h + 8 * p : 32 + 16 * h + 8 * (p - 2)) + (i >> 1);
        v[p] = __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_i2)(&Bs[16 * ldsB(kr, c) + 8 * (i & 1)]));
      }
    } else {
      // ds_read_b64_tr_b16: lane i of a 16-lane group addresses row i/4,
      // columns 4 (i%4).. of a 4 x 16 block and receives column i; two
      // reads per 8 k (rows 8h.. and 8h + 4..), k 16.. for the second MFMA
      const int n = wn * WTN + 32 * ni + 16 * (q & 1) + 4 * (i & 3);
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const int kr = 16 * (p >> 1) + 8 * h + 4 * (p & 1) + (i >> 2);
        v[p] = __builtin_bit_cast(intx2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                                             (lds_s4)(&Bs[16 * ldsB(kr, n / 8) + 2 * (n % 8)])));
      }
    }
    f = intx8{v[0][0], v[0][1], v[1][0], v[1][1], v[2][0], v[2][1], v[3][0], v[3][1]};
  };

  // prologue: slabs 0 .. D-1 issued, 0 and 1 landed (all waves), slab 0's
  // fragments read
  static_for<0, D>([&](auto x) { static_for<0, NI>([&](auto t) { dma1(x, x, t); }); });
  __builtin_amdgcn_s_waitcnt(vmcnt_only((D - 2) * NI));
  barrier_nofence();
  constexpr std::integral_constant<int, 0> S0{};
#pragma unroll
  for (int mi = 0; mi < TM; ++mi) rdA(S0, mi, fa[0][mi]);
#pragma unroll
  for (int ni = 0; ni < TN; ++ni) rdB(S0, ni, fb[0][ni]);
  lds_wait();
  barrier_nofence();

  auto step = [&](int sl, auto X_) {
    constexpr int x = decltype(X_)::value, cur = x & 1, nxt = cur ^ 1;
    constexpr std::integral_constant<int, (x + 1) % NS> rslot{};
    constexpr std::integral_constant<int, (x + D) % NS> wslot{};
    __builtin_amdgcn_sched_barrier(0);
    static_for<0, TM>([&](auto mi) {
#pragma unroll
      for (int ni = 0; ni < TN; ++ni) {
        if constexpr (EB == 1) {
          acc[mi][ni] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(fa[cur][mi], fb[cur][ni], acc[mi][ni],
                                                                        0, 0, 0, 127, 0, 127);
        } else {
          const intx8& x = fa[0][mi];
          const intx8& y = fb[cur][ni];
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8, __builtin_shufflevector(x, x, 0, 1, 2, 3)),
              __builtin_bit_cast(bf16x8, __builtin_shufflevector(y, y, 0, 1, 2, 3)), acc[mi][ni], 0, 0, 0);
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8, __builtin_shufflevector(x, x, 4, 5, 6, 7)),
              __builtin_bit_cast(bf16x8, __builtin_shufflevector(y, y, 4, 5, 6, 7)), acc[mi][ni], 0, 0, 0);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      constexpr int MI = decltype(mi)::value;
      rdA(rslot, MI, fa[FA == 1 ? 0 : nxt][MI]);
      if constexpr (MI < TN) rdB(rslot, MI, fb[nxt][MI]);
      // the step's NI loads spread over the TM row groups
      static_for<0, NI>([&](auto t) {
        if constexpr (decltype(t)::value * TM / NI == MI) dma1(sl + D, wslot, t);
      });
      __builtin_amdgcn_sched_barrier(0);
    });
    lds_wait();
    __builtin_amdgcn_s_waitcnt(vmcnt_only((D - 2) * NI));   // the wave's loads of slab sl+2 landed
    barrier_nofence();
  };
  // slot x % NS, fragment set x & 1: the pattern repeats every U slabs.
  // Whole groups of U run unguarded; the last group stops at the part end
  // (slabs past it would be zero: no product, accumulators unchanged)
  constexpr int U = NS % 2 == 0 ? NS : 2 * NS;
  int sl = 0;
  for (; sl + U <= nslab; sl += U)
    static_for<0, U>([&](auto x) { step(sl + x, x); });
  if (sl < nslab)
    static_for<0, U>([&](auto x) {
      if (sl + decltype(x)::value < nslab) step(sl + x, x);
    });
  __builtin_amdgcn_s_waitcnt(vmcnt_only(0));   // nothing lands in the staging area later
  __syncthreads();

  // epilogue: the block's bias as binary32 in the B array of slot 0; wave
  // w stages 16-row halves of its 32-row bands through its own A array
  // (pitch WTN + 8 floats: the two row sets of one write sit 32 banks
  // apart) and finishes four columns per store, two stores in flight
  constexpr int CSP = WTN + 8;
  static_assert(16 * CSP * 4 <= 16384 && BN * 4 <= B_BYTES, "epilogue staging fits");
  float* bsh = reinterpret_cast<float*>(f8w_bslot<BN, 0>());
  stage_bias(a, j0, BN, bsh);
  __syncthreads();
  const bool bias = needs_bias(a);
  // (256 x 128 blocks: two waves per A array, 8 KB each, within the ring's three)
  float* cs = BN == 256 ? reinterpret_cast<float*>(wave == 0 ? f8w_a0 : wave == 1 ? f8w_a1 : wave == 2 ? f8w_a2 : f8w_a3)
                        : reinterpret_cast<float*>((wave < 2 ? f8w_a0 : f8w_a1) + 8192 * (wave & 1));
  static_assert(BN == 256 || 16 * CSP * 4 <= 8192, "two staging areas per A array");
#pragma unroll
  for (int mi = 0; mi < TM; ++mi) {
#pragma unroll
    for (int half = 0; half < 2; ++half) {
#pragma unroll
      for (int ni = 0; ni < TN; ++ni)
#pragma unroll
        for (int r = 8 * half; r < 8 * half + 8; ++r)
          cs[(8 * (r / 4) - 16 * half + 4 * (lane >> 5) + (r & 3)) * CSP + 32 * ni + (lane & 31)] = acc[mi][ni][r];
      lds_wait();
#pragma unroll 2
      for (int q = lane; q < 16 * WTN / 4; q += 64) {
        const int rr = q / (WTN / 4), cc = 4 * (q % (WTN / 4));
        const int64_t gi = i0 + wm * WTM + 32 * mi + 16 * half + rr, gj = j0 + wn * WTN + cc;
        const float4 b4 = bias ? *(const float4*)&bsh[wn * WTN + cc] : float4{0.f, 0.f, 0.f, 0.f};
        if (gi < a.M && gj < a.N) (void)finish4v(a, s, gi, gj, *(const float4*)&cs[rr * CSP + cc], b4);
      }
      lds_wait();
    }
  }
}

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void gemm_f8w(GemmArgs a) {
  const int tiles_m = (int)((a.M + 255) / 256);
  int ty, tx;
  grouped_tile(blockIdx.x, tiles_m, gridDim.x / tiles_m, a.order, &ty, &tx);
  f8w_body<256>(a, (int64_t)ty * 256, (int64_t)tx * 256);
}

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void gemm_f8n(GemmArgs a) {
  const int tiles_m = (int)((a.M + 255) / 256);
  int ty, tx;
  grouped_tile(blockIdx.x, tiles_m, gridDim.x / tiles_m, a.order, &ty, &tx);
  f8w_body<128>(a, (int64_t)ty * 256, (int64_t)tx * 128);
}

// bf16 operands on the same pipeline (256 x 128 blocks, two per CU).
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void gemm_b16n(GemmArgs a) {
  const int tiles_m = (int)((a.M + 255) / 256);
  int ty, tx;
  grouped_tile(blockIdx.x, tiles_m, gridDim.x / tiles_m, a.order, &ty, &tx);
  f8w_body<128, 2>(a, (int64_t)ty * 256, (int64_t)tx * 128);
}

// Columns [0, n_split) in 256 x 256 blocks, the rest in 256 x 192 blocks.
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void gemm_w4_mixed(GemmArgs a) {
  const int tiles_m = (int)((a.M + 255) / 256);
  const int tn1 = (int)((a.n_split + 255) / 256), nb1 = tiles_m * tn1;
  int ty, tx;
  if ((int)blockIdx.x < nb1) {
    grouped_tile(blockIdx.x, tiles_m, tn1, a.order, &ty, &tx);
    w4d_body<256>(a, (int64_t)ty * 256, (int64_t)tx * 256);
  } else {
    const int tn2 = a.N > a.n_split ? (int)((a.N - a.n_split + 191) / 192) : 0;
    grouped_tile(blockIdx.x - nb1, tiles_m, tn2, a.order, &ty, &tx);
    w4d_body<192>(a, (int64_t)ty * 256, a.n_split + (int64_t)tx * 192);
  }
}

// ---------------------------------------------------------- skinny (M <= 64)
//
// Few rows: the GEMM streams B from HBM and the MFMA work per slab is small,
// so the time goes to memory latency.  Each workgroup owns BN columns (one
// 16-column MFMA tile per computing wave, all four waves loading) and keeps
// D BK-k slabs of loads in flight through a ring of D register sets, staged
// through an LDS double buffer in the layouts of the v3 kernel (A [m][k], B
// [k][n], transposing reads for B).  Same chunk order as every other path.
// When the column tiles split evenly over the eight XCDs (workgroup w runs
// on XCD w mod 8), each XCD takes a contiguous range of them, so that tiles
// sharing 128-byte B lines share an L2.
template <int TMS, int BN, int D, int BK, bool F16>
__global__ __launch_bounds__(256) void gemm_skinny(GemmArgs a) {
  constexpr int CPR = BK / 8, BM = 16 * TMS, NWC = BN / 16;
  constexpr int ACH = BM * CPR, BCH = BK * (BN / 8), BROW = BN / 8;
  constexpr int ACH_T = (ACH + 255) / 256, BCH_T = (BCH + 255) / 256;
  constexpr int A_ELEMS = BM * BK, B_ELEMS = BK * BN;
  static_assert(BN % 64 == 0 || BN == 16 || BN == 32, "B rows of whole swizzle blocks");
  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * (A_ELEMS + B_ELEMS)];
  uint16_t* As0 = smem;
  uint16_t* Bs0 = smem + 2 * A_ELEMS;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nt = gridDim.x, x = blockIdx.x;
  const int tile = (nt % 8 == 0) ? (x % 8) * (nt / 8) + x / 8 : x;
  const int64_t i0 = (int64_t)blockIdx.y * BM, j0 = (int64_t)tile * BN;
  const int s = blockIdx.z;
  // slab sl of the part covers [k0 + sl kstep, + BK), loads stop at k1: a
  // contiguous part steps by BK through [cuts[s], cuts[s+1]); a strided part
  // (dealt tiles of width BK) steps by S BK from s BK up to K
  const bool strided = a.split_w != 0;
  const int64_t k0 = strided ? (int64_t)s * BK : a.cuts[s];
  const int64_t k1 = strided ? a.K : a.cuts[s + 1];
  const int64_t kstep = strided ? (int64_t)a.S * BK : BK;
  const int nslab = (k1 > k0) ? (int)((k1 - k0 + kstep - 1) / kstep) : 0;
  static_assert(CPR >= 8, "A rows of whole swizzle blocks");
  auto ldsA = [](int row, int c) { return row * CPR + (c ^ ((row >> 1) & 7)); };
  // rows of fewer than 8 chunks (BN < 64) are swizzled within the row
  auto ldsB = [](int k, int c) { return k * BROW + ((c ^ ((k & 3) << 1)) & (BROW - 1)); };

  u32x4 ra[D][ACH_T], rb[D][BCH_T];
  auto gload = [&](int sl, u32x4* xa, u32x4* xb) {
    const int64_t ks = k0 + (int64_t)sl * kstep;
#pragma unroll
    for (int t = 0; t < ACH_T; ++t) {
      const int q = tid + 256 * t, row = q / CPR, c = q % CPR;
      const int64_t gi = i0 + row, gk = ks + 8 * c;
      xa[t] = *chunk_or_zero((q < ACH) && (gi < a.M) && (gk < k1), a.A + gi * a.K + gk);
    }
#pragma unroll
    for (int t = 0; t < BCH_T; ++t) {
      const int q = tid + 256 * t, kr = q / BROW, c = q % BROW;
      const int64_t gk = ks + kr, gn = j0 + 8 * c;
      xb[t] = *chunk_or_zero((q < BCH) && (gk < k1) && (gn < a.N), a.B + gk * a.N + gn);
    }
  };
  auto lstore = [&](int buf, const u32x4* xa, const u32x4* xb) {
    uint16_t* As = As0 + buf * A_ELEMS;
    uint16_t* Bs = Bs0 + buf * B_ELEMS;
#pragma unroll
    for (int t = 0; t < ACH_T; ++t) {
      const int q = tid + 256 * t;
      if (q < ACH) *(u32x4*)&As[8 * ldsA(q / CPR, q % CPR)] = xa[t];
    }
#pragma unroll
    for (int t = 0; t < BCH_T; ++t) {
      const int q = tid + 256 * t;
      if (q < BCH) *(u32x4*)&Bs[8 * ldsB(q / BROW, q % BROW)] = xb[t];
    }
  };
  floatx4 acc[TMS];
#pragma unroll
  for (int mi = 0; mi < TMS; ++mi) acc[mi] = floatx4{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](int buf) {
    if (wave >= NWC) return;
    const uint16_t* As = As0 + buf * A_ELEMS;
    const uint16_t* Bs = Bs0 + buf * B_ELEMS;
#pragma unroll
    for (int kk = 0; kk < BK; kk += 32) {
      const int i = lane & 15, g = lane >> 4;
      const int n = 16 * wave + 4 * (i & 3);
      const int kr0 = kk + 8 * g + (i >> 2), kr1 = kr0 + 4;
      const shortx4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)(&Bs[8 * ldsB(kr0, n / 8) + (n & 7)]));
      const shortx4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)(&Bs[8 * ldsB(kr1, n / 8) + (n & 7)]));
      const shortx8 bfr = shortx8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
#pragma unroll
      for (int mi = 0; mi < TMS; ++mi) {
        const shortx8 af = *(const shortx8*)&As[8 * ldsA(16 * mi + (lane & 15), kk / 8 + (lane >> 4))];
        acc[mi] = mfma16t<F16>(af, bfr, acc[mi]);
      }
    }
  };

  // Loads and LDS stores are issued unconditionally (a slab past the part
  // end reads the zero chunk), so that every path holds the same number of
  // loads in flight and the LDS store of slab s+1 waits only for its own
  // loads, not for the D-1 slabs behind it.  Only the MFMA work is skipped.
  static_for<0, D>([&](auto j) { gload(j, ra[j], rb[j]); });
  lstore(0, ra[0], rb[0]);
  __syncthreads();
  for (int base = 0; base < nslab; base += D) {
    static_for<0, D>([&](auto u) {
      const int sl = base + u;
      if (sl < nslab) compute(sl & 1);
      gload(sl + D, ra[u], rb[u]);
      lstore((sl + 1) & 1, ra[(u + 1) % D], rb[(u + 1) % D]);
      __syncthreads();
    });
  }
  if (wave < NWC) {
#pragma unroll
    for (int mi = 0; mi < TMS; ++mi)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t i = i0 + 16 * mi + 4 * (lane >> 4) + r, j = j0 + 16 * wave + (lane & 15);
        if (i < a.M && j < a.N) finish(a, s, i, j, acc[mi][r]);
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

template <int MR, int CPT>
static void launch_scalar_t(const GemmArgs& a, hipStream_t st) {
  dim3 grid((unsigned)((a.N + 256 * CPT - 1) / (256 * CPT)), (unsigned)((a.M + MR - 1) / MR), (unsigned)a.S);
  if (a.in_f16) hipLaunchKernelGGL((gemm_scalar<MR, CPT, true>), grid, dim3(256), 0, st, a);
  else hipLaunchKernelGGL((gemm_scalar<MR, CPT, false>), grid, dim3(256), 0, st, a);
}

hipError_t launch_gemm_scalar(const GemmArgs& a, hipStream_t st) {
  const int mr = a.M >= 4 ? 4 : a.M >= 2 ? 2 : 1;
  // four columns per thread (one 8-byte load per row of B) when rows allow it
  const bool vec = a.N % 4 == 0 && ((uintptr_t)a.B) % 8 == 0;
  if (vec) {
    if (mr == 4) launch_scalar_t<4, 4>(a, st);
    else if (mr == 2) launch_scalar_t<2, 4>(a, st);
    else launch_scalar_t<1, 4>(a, st);
  } else {
    if (mr == 4) launch_scalar_t<4, 1>(a, st);
    else if (mr == 2) launch_scalar_t<2, 1>(a, st);
    else launch_scalar_t<1, 1>(a, st);
  }
  return hipGetLastError();
}

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

template <int BM, int BN, int WM, int WN>
static hipError_t launch_big_t(const GemmArgs& a, hipStream_t st) {
  const int64_t tm = (a.M + BM - 1) / BM, tn = (a.N + BN - 1) / BN;
  hipLaunchKernelGGL((gemm_big<BM, BN, WM, WN>), dim3((unsigned)(tm * tn), 1, (unsigned)a.S), dim3(256), 0, st, a);
  return hipGetLastError();
}

template <int BM, int BN, int WM, int WN, int BK, bool TWO>
static hipError_t launch_v3_t(const GemmArgs& a, hipStream_t st) {
  const int64_t tm = (a.M + BM - 1) / BM, tn = (a.N + BN - 1) / BN;
  dim3 grid((unsigned)(tm * tn), 1, (unsigned)a.S);
  if (a.in_f16) {
    if constexpr (TWO) hipLaunchKernelGGL((gemm_v3x2<BM, BN, WM, WN, BK, true>), grid, dim3(256), 0, st, a);
    else hipLaunchKernelGGL((gemm_v3<BM, BN, WM, WN, BK, true>), grid, dim3(256), 0, st, a);
  } else {
    if constexpr (TWO) hipLaunchKernelGGL((gemm_v3x2<BM, BN, WM, WN, BK, false>), grid, dim3(256), 0, st, a);
    else hipLaunchKernelGGL((gemm_v3<BM, BN, WM, WN, BK, false>), grid, dim3(256), 0, st, a);
  }
  return hipGetLastError();
}

template <int BM, int BN, int BK>
static hipError_t launch_pp_t(const GemmArgs& a, hipStream_t st) {
  const int64_t tm = (a.M + BM - 1) / BM, tn = (a.N + BN - 1) / BN;
  if (a.in_f16) hipLaunchKernelGGL((gemm_pp<BM, BN, BK, true>), dim3((unsigned)(tm * tn), 1, (unsigned)a.S), dim3(512), 0, st, a);
  else hipLaunchKernelGGL((gemm_pp<BM, BN, BK, false>), dim3((unsigned)(tm * tn), 1, (unsigned)a.S), dim3(512), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_gemm_pp_mixed(const GemmArgs& a, hipStream_t st) {
  const int64_t tm = (a.M + 255) / 256, tn = a.n_split / 256 + (a.N - a.n_split + 191) / 192;
  if (a.in_f16) hipLaunchKernelGGL((gemm_pp_mixed<32, true>), dim3((unsigned)(tm * tn), 1, (unsigned)a.S), dim3(512), 0, st, a);
  else hipLaunchKernelGGL((gemm_pp_mixed<32, false>), dim3((unsigned)(tm * tn), 1, (unsigned)a.S), dim3(512), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_gemm_w4(const GemmArgs& a, hipStream_t st) {
  const int64_t tm = (a.M + 255) / 256, tn = (a.n_split + 255) / 256 + (a.N > a.n_split ? (a.N - a.n_split + 191) / 192 : 0);
  hipLaunchKernelGGL(gemm_w4_mixed, dim3((unsigned)(tm * tn), 1, (unsigned)a.S), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_gemm_ppd(const GemmArgs& a, bool mixed, hipStream_t st) {
  const int64_t tm = (a.M + 255) / 256;
  if (mixed) {
    const int64_t tn = a.n_split / 256 + (a.N - a.n_split + 191) / 192;
    hipLaunchKernelGGL(gemm_ppd_mixed, dim3((unsigned)(tm * tn), 1, (unsigned)a.S), dim3(512), 0, st, a);
  } else {
    const int64_t tn = (a.N + 255) / 256;
    hipLaunchKernelGGL(gemm_ppd, dim3((unsigned)(tm * tn), 1, (unsigned)a.S), dim3(512), 0, st, a);
  }
  return hipGetLastError();
}

bool wide_supported(int tm, int tn) {
  return (tm == 256 || tm == 128) && (tn == 256 || tn == 128);
}

bool wide_is_pp(int tm, int tn) { return wide_supported(tm, tn); }

hipError_t launch_gemm_wide(const GemmArgs& a, int tm, int tn, hipStream_t st) {
  if (tm == 256 && tn == 256) return launch_pp_t<256, 256, 32>(a, st);
  if (tm == 256 && tn == 128) return launch_pp_t<256, 128, 64>(a, st);
  if (tm == 128 && tn == 256) return launch_pp_t<128, 256, 64>(a, st);
  if (tm == 128 && tn == 128) return launch_pp_t<128, 128, 64>(a, st);
  return hipErrorInvalidValue;
}

// ------------------------------------------ few rows, direct-to-LDS ring
//
// The few-row kernel's order and LDS layouts, with the slabs loaded from
// memory straight into a ring of NS LDS slots (separate arrays, so that the
// compiler waits only for the slot it reads) instead of through registers:
// NS - 1 slabs stay in flight per workgroup, limited by LDS rather than by
// registers, which is what a B stream from HBM needs.  One barrier per slab:
// a thread waits until its loads of slab s have landed, the barrier makes
// every thread's visible, the slab is computed, and the loads of slab
// s + NS - 1 go into the slot slab s - 1 left (free once every thread has
// passed this barrier).  Each load instruction fills 1 KB of a slot with the
// lanes in layout order; each lane fetches the chunk the swizzle puts there.
template <int TMS, int BN, int NS, int BK>
__global__ __launch_bounds__(256) void gemm_skinny_dma(GemmArgs a) {
  constexpr int CPR = BK / 8, BM = 16 * TMS, NWC = BN / 16, BROW = BN / 8;
  constexpr int A_ELEMS = BM * BK, B_ELEMS = BK * BN, SLOT = A_ELEMS + B_ELEMS;
  constexpr int NA = BM * BK / 2048, NB = BK * BN / 2048;      // 1 KB loads per wave per slab
  constexpr int ND = NA + NB;
  static_assert(NA >= 1 && NB >= 1 && BM * BK % 2048 == 0 && BK * BN % 2048 == 0, "whole 1 KB loads per wave");
  static_assert(CPR >= 8 && (BN == 16 || BN == 32 || BN == 64), "layouts of the few-row kernel");
  static_assert(NS >= 3 && NS <= 8, "ring depth");
  __shared__ __attribute__((aligned(1024))) uint16_t q0[SLOT], q1[SLOT], q2[SLOT], q3[SLOT];
  __shared__ __attribute__((aligned(1024))) uint16_t q4[NS > 4 ? SLOT : 8], q5[NS > 5 ? SLOT : 8];
  __shared__ __attribute__((aligned(1024))) uint16_t q6[NS > 6 ? SLOT : 8], q7[NS > 7 ? SLOT : 8];
  auto slot = [&](auto S) -> uint16_t* {
    constexpr int i = decltype(S)::value;
    if constexpr (i == 0) return q0;
    else if constexpr (i == 1) return q1;
    else if constexpr (i == 2) return q2;
    else if constexpr (i == 3) return q3;
    else if constexpr (i == 4) return q4;
    else if constexpr (i == 5) return q5;
    else if constexpr (i == 6) return q6;
    else return q7;
  };
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nt = gridDim.x, x = blockIdx.x;
  const int tile = (nt % 8 == 0) ? (x % 8) * (nt / 8) + x / 8 : x;
  const int64_t i0 = (int64_t)blockIdx.y * BM, j0 = (int64_t)tile * BN;
  const int s = blockIdx.z;
  const bool strided = a.split_w != 0;
  const int64_t k0 = strided ? (int64_t)s * BK : a.cuts[s];
  const int64_t k1 = strided ? a.K : a.cuts[s + 1];
  const int64_t kstep = strided ? (int64_t)a.S * BK : BK;
  const int nslab = (k1 > k0) ? (int)((k1 - k0 + kstep - 1) / kstep) : 0;
  auto ldsA = [](int row, int c) { return row * CPR + (c ^ ((row >> 1) & 7)); };
  auto ldsB = [](int k, int c) { return k * BROW + ((c ^ ((k & 3) << 1)) & (BROW - 1)); };

  constexpr uint32_t OOB = 0x80000000u;
  const int64_t recA = (a.M - i0) * a.K * 2, recB = a.K * a.N * 2;
  const __amdgpu_buffer_rsrc_t rA = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a.A + i0 * a.K), (short)0, (int)(recA < 0x7fffffff ? recA : 0x7fffffff), 0x00020000);
  const __amdgpu_buffer_rsrc_t rB = __builtin_amdgcn_make_buffer_rsrc(
      (void*)a.B, (short)0, (int)(recB < 0x7fffffff ? recB : 0x7fffffff), 0x00020000);
  // load t of the wave: A runs first (64 / CPR rows per KB), then B runs
  // (64 / BROW k-rows per KB); lane l holds the run's l-th 16-byte slot
  uint32_t off[ND];
  int kc[ND], dst[ND];
#pragma unroll
  for (int t = 0; t < ND; ++t) {
    const int run = wave * ND + t;   // runs 0 .. 4 ND - 1 of the slab: 4 NA of A, then 4 NB of B
    if (run < 4 * NA) {
      const int row = run * (64 / CPR) + lane / CPR, pc = lane % CPR;
      const int c = pc ^ ((row >> 1) & 7);
      off[t] = (i0 + row < a.M) ? (uint32_t)((row * a.K + 8 * c) * 2) : OOB;
      kc[t] = 8 * c;
      dst[t] = 8 * ldsA(row, c) - 8 * lane;   // the run's first element (lanes in layout order)
    } else {
      const int rb = run - 4 * NA;
      const int kr = rb * (64 / BROW) + lane / BROW, pc = lane % BROW;
      const int c = (pc ^ ((kr & 3) << 1)) & (BROW - 1);
      off[t] = (j0 + 8 * c < a.N) ? (uint32_t)((kr * a.N + j0 + 8 * c) * 2) : OOB;
      kc[t] = kr;
      dst[t] = A_ELEMS + 8 * ldsB(kr, c) - 8 * lane;
    }
  }
  auto dma = [&](auto S, int sl) {
    uint16_t* base = slot(S);
    const int64_t ks = k0 + (int64_t)sl * kstep, lim = k1 - ks;
#pragma unroll
    for (int t = 0; t < ND; ++t) {
      const uint32_t o = kc[t] < lim ? off[t] : OOB;
      const int d = __builtin_amdgcn_readfirstlane(dst[t]);
      if (wave * ND + t < 4 * NA)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rA, (lds_void)(base + d), 16, o, (int)(ks * 2), 0, 0);
      else
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rB, (lds_void)(base + d), 16, o, (int)(ks * a.N * 2), 0, 0);
    }
  };
  floatx4 acc[TMS];
#pragma unroll
  for (int mi = 0; mi < TMS; ++mi) acc[mi] = floatx4{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](auto S) {
    if (wave >= NWC) return;
    const uint16_t* As = slot(S);
    const uint16_t* Bs = As + A_ELEMS;
#pragma unroll
    for (int kk = 0; kk < BK; kk += 32) {
      const int i = lane & 15, g = lane >> 4;
      const int n = 16 * wave + 4 * (i & 3);
      const int kr0 = kk + 8 * g + (i >> 2), kr1 = kr0 + 4;
      const shortx4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)(&Bs[8 * ldsB(kr0, n / 8) + (n & 7)]));
      const shortx4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)(&Bs[8 * ldsB(kr1, n / 8) + (n & 7)]));
      const shortx8 bfr = shortx8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
#pragma unroll
      for (int mi = 0; mi < TMS; ++mi) {
        const shortx8 af = *(const shortx8*)&As[8 * ldsA(16 * mi + (lane & 15), kk / 8 + (lane >> 4))];
        acc[mi] = mfma16(af, bfr, acc[mi]);
      }
    }
  };
  // prologue: slabs 0 .. NS-2 in flight
  static_for<0, NS - 1>([&](auto u) { dma(u, u); });
  for (int base = 0; base < nslab; base += NS) {
    static_for<0, NS>([&](auto u) {
      const int sl = base + u;
      __builtin_amdgcn_s_waitcnt(vmcnt_only((NS - 2) * ND));   // slab sl landed
      barrier_nofence();
      if (sl < nslab) compute(u);
      dma(std::integral_constant<int, (u + NS - 1) % NS>{}, sl + NS - 1);
    });
  }
  __builtin_amdgcn_s_waitcnt(vmcnt_only(0));
  if (wave < NWC) {
#pragma unroll
    for (int mi = 0; mi < TMS; ++mi)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t i = i0 + 16 * mi + 4 * (lane >> 4) + r, j = j0 + 16 * wave + (lane & 15);
        if (i < a.M && j < a.N) finish(a, s, i, j, acc[mi][r]);
      }
  }
}

template <int TMS, int BN, int NS, int BK>
static hipError_t launch_skinny_dma_t(const GemmArgs& a, hipStream_t st) {
  dim3 grid((unsigned)((a.N + BN - 1) / BN), (unsigned)((a.M + 16 * TMS - 1) / (16 * TMS)), (unsigned)a.S);
  hipLaunchKernelGGL((gemm_skinny_dma<TMS, BN, NS, BK>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

// (tile_m, tile_n, ring slots, slab_k) combinations built
#define DG_SKINNY_DMA_LIST(X) \
  X(16, 16, 4, 256) X(16, 16, 8, 256) X(16, 32, 4, 256) X(16, 32, 6, 256) X(32, 32, 4, 128) X(32, 32, 6, 128) \
  X(64, 32, 4, 128) X(64, 32, 3, 128) X(16, 64, 4, 128) X(16, 64, 6, 128)

bool skinny_dma_supported(int tm, int tn, int slots, int slab_k) {
#define DG_SKDMA_HAS(TM_, TN_, NS_, BK_) \
  if (tm == TM_ && tn == TN_ && slots == NS_ && slab_k == BK_) return true;
  DG_SKINNY_DMA_LIST(DG_SKDMA_HAS)
#undef DG_SKDMA_HAS
  return false;
}

hipError_t launch_gemm_skinny_dma(const GemmArgs& a, int tm, int tn, int slots, int slab_k, hipStream_t st) {
#define DG_SKDMA_RUN(TM_, TN_, NS_, BK_) \
  if (tm == TM_ && tn == TN_ && slots == NS_ && slab_k == BK_) return launch_skinny_dma_t<TM_ / 16, TN_, NS_, BK_>(a, st);
  DG_SKINNY_DMA_LIST(DG_SKDMA_RUN)
#undef DG_SKDMA_RUN
  return hipErrorInvalidValue;
}

template <int TMS, int BN, int D, int BK>
static hipError_t launch_skinny_t(const GemmArgs& a, hipStream_t st) {
  dim3 grid((unsigned)((a.N + BN - 1) / BN), (unsigned)((a.M + 16 * TMS - 1) / (16 * TMS)), (unsigned)a.S);
  if (a.in_f16) hipLaunchKernelGGL((gemm_skinny<TMS, BN, D, BK, true>), grid, dim3(256), 0, st, a);
  else hipLaunchKernelGGL((gemm_skinny<TMS, BN, D, BK, false>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

// (tile_m, tile_n, depth, slab_k) combinations built; slab_k 0 means 64
#define DG_SKINNY_LIST(X)                                                                   \
  X(16, 16, 4, 64) X(16, 16, 8, 64) X(16, 32, 4, 64) X(16, 32, 8, 64) X(16, 64, 4, 64)      \
  X(16, 64, 8, 64) X(32, 16, 4, 64) X(32, 32, 4, 64) X(32, 32, 8, 64) X(32, 64, 4, 64)      \
  X(64, 16, 4, 64) X(64, 32, 4, 64) X(64, 32, 8, 64) X(64, 64, 4, 64)                       \
  X(16, 16, 2, 256) X(16, 16, 4, 256) X(16, 32, 2, 256) X(16, 32, 4, 256) X(16, 64, 2, 256) \
  X(16, 64, 4, 256) X(32, 32, 2, 256) X(32, 64, 2, 256) X(64, 32, 2, 128) X(64, 32, 4, 128) \
  X(64, 64, 2, 128) X(16, 16, 4, 128) X(16, 32, 4, 128) X(16, 64, 4, 128) X(32, 32, 4, 128) \
  X(32, 64, 4, 128)

bool skinny_supported(int tm, int tn, int depth, int slab_k) {
  if (depth == 0) depth = 4;
  if (slab_k == 0) slab_k = 64;
#define DG_SKINNY_HAS(TM_, TN_, D_, BK_) \
  if (tm == TM_ && tn == TN_ && depth == D_ && slab_k == BK_) return true;
  DG_SKINNY_LIST(DG_SKINNY_HAS)
#undef DG_SKINNY_HAS
  return false;
}

hipError_t launch_gemm_skinny(const GemmArgs& a, int tm, int tn, int depth, int slab_k, hipStream_t st) {
  if (depth == 0) depth = 4;
  if (slab_k == 0) slab_k = 64;
#define DG_SKINNY_RUN(TM_, TN_, D_, BK_) \
  if (tm == TM_ && tn == TN_ && depth == D_ && slab_k == BK_) return launch_skinny_t<TM_ / 16, TN_, D_, BK_>(a, st);
  DG_SKINNY_LIST(DG_SKINNY_RUN)
#undef DG_SKINNY_RUN
  return hipErrorInvalidValue;
}

bool v3_supported(int tm, int tn, int occ) {
  if (occ == 2) return (tm == 128 && tn == 128) || (tm == 64 && tn == 128) || (tm == 32 && tn == 128);
  // No 256 x 256 block: its 256 accumulator registers and 64 ring registers per
  // lane leave the fragments no room, and the register spills that shape needs
  // were compiled into code that dropped the fourth dword of a spilled
  // 16-byte load (wrong bits in the block's last 64 rows).  Every shape kept
  // here compiles without spills.
  return (tm == 256 && tn == 128) || (tm == 128 && tn == 256) ||
         (tm == 128 && tn == 128) || (tm == 64 && tn == 128) || (tm == 32 && tn == 256) ||
         (tm == 32 && tn == 128);
}

hipError_t launch_gemm_v3(const GemmArgs& a, int tm, int tn, int occ, hipStream_t st) {
  if (occ == 2) {
    if (tm == 128 && tn == 128) return launch_v3_t<128, 128, 2, 2, 32, true>(a, st);
    if (tm == 64 && tn == 128) return launch_v3_t<64, 128, 2, 2, 64, true>(a, st);
    if (tm == 32 && tn == 128) return launch_v3_t<32, 128, 1, 4, 64, true>(a, st);
    return hipErrorInvalidValue;
  }
  if (tm == 256 && tn == 128) return launch_v3_t<256, 128, 2, 2, 32, false>(a, st);
  if (tm == 128 && tn == 256) return launch_v3_t<128, 256, 2, 2, 32, false>(a, st);
  if (tm == 128 && tn == 128) return launch_v3_t<128, 128, 2, 2, 64, false>(a, st);
  if (tm == 64 && tn == 128) return launch_v3_t<64, 128, 2, 2, 64, false>(a, st);
  if (tm == 32 && tn == 256) return launch_v3_t<32, 256, 1, 4, 64, false>(a, st);
  if (tm == 32 && tn == 128) return launch_v3_t<32, 128, 1, 4, 64, false>(a, st);
  return hipErrorInvalidValue;
}

template <int COMB, bool FMA0, int L>
static hipError_t launch_tc_t(const GemmArgs& a, hipStream_t st) {
  constexpr int BN = tc_bn<COMB, L>();
  const int64_t tm = (a.M + 127) / 128, tn = (a.N + BN - 1) / BN;
  dim3 grid((unsigned)(tm * tn), 1, (unsigned)a.S);
  if (a.in_f16) hipLaunchKernelGGL((gemm_tc<COMB, FMA0, L, true>), grid, dim3(256), 0, st, a);
  else hipLaunchKernelGGL((gemm_tc<COMB, FMA0, L, false>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_gemm_tc(const GemmArgs& a, int levels, hipStream_t st) {
  const bool fma0 = a.fma == 0;
  if (a.tile_combine == DG_CARRY) return fma0 ? launch_tc_t<DG_CARRY, true, 1>(a, st) : hipErrorInvalidValue;
  if (a.tile_combine == DG_SEQ) return fma0 ? launch_tc_t<DG_SEQ, true, 1>(a, st) : launch_tc_t<DG_SEQ, false, 1>(a, st);
  if (a.tile_combine != DG_TREE) return hipErrorInvalidValue;
  switch (levels) {
    case 2: return fma0 ? launch_tc_t<DG_TREE, true, 2>(a, st) : launch_tc_t<DG_TREE, false, 2>(a, st);
    case 3: return fma0 ? launch_tc_t<DG_TREE, true, 3>(a, st) : launch_tc_t<DG_TREE, false, 3>(a, st);
    case 4: return fma0 ? launch_tc_t<DG_TREE, true, 4>(a, st) : launch_tc_t<DG_TREE, false, 4>(a, st);
    case 5: return fma0 ? launch_tc_t<DG_TREE, true, 5>(a, st) : launch_tc_t<DG_TREE, false, 5>(a, st);
    case 6: return fma0 ? launch_tc_t<DG_TREE, true, 6>(a, st) : launch_tc_t<DG_TREE, false, 6>(a, st);
    case 7: return fma0 ? launch_tc_t<DG_TREE, true, 7>(a, st) : launch_tc_t<DG_TREE, false, 7>(a, st);
    default: return hipErrorInvalidValue;
  }
}

bool tiled_supported(int tm, int tn) {
  return (tm == 16 && (tn == 64 || tn == 128)) || (tm == 32 && tn == 128) ||
         (tm == 64 && tn == 128) || (tm == 128 && tn == 128) || (tm == 256 && tn == 256) ||
         (tm == 256 && tn == 128) || (tm == 128 && tn == 256);
}

hipError_t launch_gemm_tiled(const GemmArgs& a, int tm, int tn, hipStream_t st) {
  if (tm == 16 && tn == 64) return launch_tiled_t<16, 64, 1, 4>(a, st);
  if (tm == 16 && tn == 128) return launch_tiled_t<16, 128, 1, 4>(a, st);
  if (tm == 32 && tn == 128) return launch_tiled_t<32, 128, 1, 4>(a, st);
  if (tm == 64 && tn == 128) return launch_tiled_t<64, 128, 2, 2>(a, st);
  if (tm == 128 && tn == 128) return launch_tiled_t<128, 128, 2, 2>(a, st);
  if (tm == 256 && tn == 256) return launch_big_t<256, 256, 2, 2>(a, st);
  if (tm == 256 && tn == 128) return launch_big_t<256, 128, 2, 2>(a, st);
  if (tm == 128 && tn == 256) return launch_big_t<128, 256, 2, 2>(a, st);
  return hipErrorInvalidValue;
}

hipError_t launch_gemm_b16n(const GemmArgs& a, hipStream_t st) {
  const int64_t tiles = ((a.M + 255) / 256) * ((a.N + 127) / 128);
  hipLaunchKernelGGL(gemm_b16n, dim3((unsigned)tiles, 1, (unsigned)a.S), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_gemm_f8(const GemmArgs& a, int tile, hipStream_t st) {
  if (tile == 256 + 128) {   // 256 x 128 blocks
    const int64_t tiles = ((a.M + 255) / 256) * ((a.N + 127) / 128);
    hipLaunchKernelGGL(gemm_f8n, dim3((unsigned)tiles, 1, (unsigned)a.S), dim3(256), 0, st, a);
    return hipGetLastError();
  }
  if (tile == 256) {
    const int64_t tiles = ((a.M + 255) / 256) * ((a.N + 255) / 256);
    hipLaunchKernelGGL(gemm_f8w, dim3((unsigned)tiles, 1, (unsigned)a.S), dim3(256), 0, st, a);
    return hipGetLastError();
  }
  if (tile != 128) return hipErrorInvalidValue;
  const int64_t tiles = ((a.M + 127) / 128) * ((a.N + 127) / 128);
  hipLaunchKernelGGL((gemm_f8<128, 128>), dim3((unsigned)tiles, 1, (unsigned)a.S), dim3(256), 0, st, a);
  return hipGetLastError();
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
