// dg_panel.hip -- few-row GEMMs on a packed B (the descriptor's order on a
// layout chosen for the memory system; the order, not the layout, fixes the
// bits, the point of the paper's Sec. 5.2 layout pass).
//
// A row-major B read in 16-column strips (one MFMA tile per wave, which is
// all the parallelism a few-row GEMM with one accumulator per output has)
// touches 32 bytes of every 8 KB row: measured on MI355X, 256 workgroups
// streaming such strips of a 4096 x 4096 bf16 B reach 1.5 TB/s with no
// arithmetic at all, against 4.0-4.7 TB/s for the same bytes read as
// contiguous runs.  The packed form (dg_pack_b) stores every 32 x 16 block
// of B -- 32 consecutive k of 16 consecutive columns -- as one 1 KB run in
// the operand layout of v_mfma_f32_16x16x32: lane l's 16 bytes are the 8
// values B[k0 + 8 (l / 16) + e][n0 + l % 16], e = 0..7.  Runs are ordered
// by column panel, then by k block; the panel's last columns and the last
// k block are zero-filled.
//
// gemm_panel: one wave per 16-column panel, split-K part and 16 TMS rows of
// A; each k block is one coalesced 1 KB load straight into the MFMA's B
// registers (no LDS), and A's fragment (16 bytes of one row per lane) is
// loaded beside it.  A ring of D blocks stays in flight in registers.  The
// chunks are walked in increasing k from the part start, as in every other
// kernel: a contiguous part is the blocks between its cut points (interior
// cuts on multiples of 32), a strided part the blocks of its dealt tiles
// (width a multiple of 32).  Blocks past the part's end hold zeros, whose
// chunks leave the accumulators unchanged.
//
// An e4m3 B (one byte per element) packs the same way into 512-byte runs
// (8 bytes per lane); the wave widens each lane's 8 values to bf16 with the
// part's conversion instruction (exact) just before the bf16 instruction, so
// the order and bits are those of the bf16 GEMM on the widened B, with half
// the bytes streamed.
#include <type_traits>

#include "dg_device.h"
#include "dg_internal.h"
#include "dg_mma.h"

namespace dg {

namespace {

constexpr uint32_t kOOB = 0x80000000u;   // a buffer offset past any record: reads zero

__device__ __forceinline__ u32x4 load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

// 8 values of one A row from k on, each checked against K (rows whose 16-byte
// runs are not 16-byte aligned: K % 8 != 0 or A itself unaligned).
__device__ __forceinline__ u32x4 load_a_elems(__amdgpu_buffer_rsrc_t r, int64_t row_off, int64_t k, int64_t K,
                                              bool row_ok) {
  uint32_t w[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint32_t o0 = (row_ok && k + 2 * e < K) ? (uint32_t)((row_off + k + 2 * e) * 2) : kOOB;
    const uint32_t o1 = (row_ok && k + 2 * e + 1 < K) ? (uint32_t)((row_off + k + 2 * e + 1) * 2) : kOOB;
    const uint32_t lo = __builtin_amdgcn_raw_buffer_load_b16(r, o0, 0, 0);
    const uint32_t hi = __builtin_amdgcn_raw_buffer_load_b16(r, o1, 0, 0);
    w[e] = (lo & 0xffffu) | (hi << 16);
  }
  return u32x4{w[0], w[1], w[2], w[3]};
}

}  // namespace

// BT: the B operand, 0 bf16, 1 binary16 (A binary16 too), 2 OCP e4m3 bytes
// (512-byte runs, widened to bf16 before the instruction)
template <int TMS, int D, bool AVEC, bool STRIDED, int BT>
__global__ __launch_bounds__(64) void gemm_panel(GemmArgs a) {
  constexpr bool F16 = BT == 1;
  constexpr int RUN = BT == 2 ? 512 : 1024;   // bytes of one block's run
  const int lane = threadIdx.x;
  const int64_t panel = blockIdx.x;
  const int64_t i0 = (int64_t)blockIdx.y * 16 * TMS, j0 = panel * 16;
  const int s = blockIdx.z;
  // every k block index and byte offset fits 31 bits (the host keeps the
  // packed B under 2 GiB and A's rows under 2 GiB)
  const int KB = (int)((a.K + 31) / 32), K = (int)a.K;
  // blocks of part s: contiguous from fb0, or dealt tiles of 2^lgw blocks
  int nf = 0, fb0 = 0, lgw = 0;
  if constexpr (STRIDED) {
    lgw = __builtin_ctz((unsigned)(a.split_w / 32));
    const int w = (int)a.split_w, ntile = (K + w - 1) / w;
    nf = ntile > s ? ((ntile - s + a.S - 1) / a.S) << lgw : 0;
  } else if (a.cuts[s + 1] > a.cuts[s]) {
    fb0 = (int)(a.cuts[s] / 32);
    nf = (int)((a.cuts[s + 1] + 31) / 32) - fb0;
  }
  const int64_t recA = (a.M - i0) * a.K * 2, recB = ((a.N + 15) / 16) * (int64_t)KB * RUN;
  const __amdgpu_buffer_rsrc_t rA = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a.A + i0 * a.K), (short)0, (int)(recA < 0x7fffffff ? recA : 0x7fffffff), 0x00020000);
  // the panel's runs: a base moved to the panel, the block in the scalar offset
  const __amdgpu_buffer_rsrc_t rB = __builtin_amdgcn_make_buffer_rsrc((void*)a.B, (short)0, (int)recB, 0x00020000);
  const int kl = 8 * (lane >> 4);   // the lane's first k within a block
  // lane constants: B's run slot; A's row run (out of range past M), and the
  // first block whose 8 k of this lane lie at or past K (only the last block
  // when K % 32 != 0).  A block's offset goes in the scalar buffer offset.
  const uint32_t vb = (uint32_t)(panel * KB * RUN) + (uint32_t)lane * (RUN / 64);
  const int flim = (K - kl + 31) / 32;
  uint32_t va[TMS];
#pragma unroll
  for (int mi = 0; mi < TMS; ++mi) {
    const int row = 16 * mi + (lane & 15);
    va[mi] = (i0 + row < a.M) ? (uint32_t)((row * K + kl) * 2) : kOOB;
  }
  // blocks q < nfe are real (a strided part's last dealt tile may run past
  // K's last block: those blocks read as zeros)
  const int nfe = STRIDED ? nf : (nf < KB - fb0 ? nf : KB - fb0);

  // block q of the part -> global k block
  auto block_of = [&](int q) -> int {
    if constexpr (STRIDED) return ((s + a.S * (q >> lgw)) << lgw) + (q & ((1 << lgw) - 1));
    else return fb0 + q;
  };
  // B's ring: 16 bytes (bf16, binary16) or 8 bytes (e4m3) per lane and block
  using BReg = std::conditional_t<BT == 2, u32x2, u32x4>;
  BReg rb[D];
  u32x4 ra[D][TMS];
  auto load = [&](int u, int q) {
    const int f = block_of(q);
    const bool ok = q < nfe && (!STRIDED || f < KB);
    const int so = ok ? f : 0;
    if constexpr (BT == 2)
      rb[u] = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(rB, ok ? vb : kOOB, so * RUN, 0));
    else
      rb[u] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rB, ok ? vb : kOOB, so * RUN, 0));
#pragma unroll
    for (int mi = 0; mi < TMS; ++mi) {
      if constexpr (AVEC) {
        ra[u][mi] = __builtin_bit_cast(
            u32x4, __builtin_amdgcn_raw_buffer_load_b128(rA, (ok && f < flim) ? va[mi] : kOOB, so * 64, 0));
      } else {
        const int row = 16 * mi + (lane & 15);
        ra[u][mi] = load_a_elems(rA, (int64_t)row * a.K, (int64_t)f * 32 + kl, a.K, ok && i0 + row < a.M);
      }
    }
  };

  floatx4 acc[TMS];
#pragma unroll
  for (int mi = 0; mi < TMS; ++mi) acc[mi] = floatx4{0.f, 0.f, 0.f, 0.f};
  // The loads stay in ring order (no scheduling across the barriers): the
  // waits count on block q's loads being older than those of q + 1.
  static_for<0, D>([&](auto u) {
    load(u, u);
    __builtin_amdgcn_sched_barrier(0);
  });
  for (int base = 0; base < nf; base += D) {
    static_for<0, D>([&](auto u) {
      const int q = base + u;
      // this block's loads are the oldest D - 1 + 1 groups in flight
      if constexpr (AVEC) __builtin_amdgcn_s_waitcnt(vmcnt_only((D - 1) * (1 + TMS)));
      if (q < nf) {
        u32x4 bw;
        if constexpr (BT == 2)
          bw = u32x4{e4m3x2_bf16x2<false>(rb[u][0]), e4m3x2_bf16x2<true>(rb[u][0]),
                     e4m3x2_bf16x2<false>(rb[u][1]), e4m3x2_bf16x2<true>(rb[u][1])};
        else
          bw = rb[u];
#pragma unroll
        for (int mi = 0; mi < TMS; ++mi)
          acc[mi] = mfma16t<F16>(__builtin_bit_cast(shortx8, ra[u][mi]), __builtin_bit_cast(shortx8, bw), acc[mi]);
      }
      load(u, q + D);
      __builtin_amdgcn_sched_barrier(0);
    });
  }
#pragma unroll
  for (int mi = 0; mi < TMS; ++mi)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t i = i0 + 16 * mi + 4 * (lane >> 4) + r, j = j0 + (lane & 15);
      if (i < a.M && j < a.N) finish(a, s, i, j, acc[mi][r]);
    }
}

// The packed form of B (K x N, 16-bit elements, row-major): thread t writes
// lane l = t % 64 of run t / 64 (panel p = run / KB, k block f = run % KB).
__global__ __launch_bounds__(256) void pack_b(const uint16_t* __restrict__ B, uint16_t* __restrict__ Bp, int64_t K,
                                              int64_t N, int64_t runs) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= runs * 64) return;
  const int64_t run = t / 64, KB = (K + 31) / 32;
  const int l = (int)(t % 64);
  const int64_t p = run / KB, f = run % KB;
  const int64_t n = p * 16 + (l & 15), k0 = f * 32 + 8 * (l >> 4);
  uint32_t w[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint32_t lo = (n < N && k0 + 2 * e < K) ? B[(k0 + 2 * e) * N + n] : 0;
    const uint32_t hi = (n < N && k0 + 2 * e + 1 < K) ? B[(k0 + 2 * e + 1) * N + n] : 0;
    w[e] = lo | (hi << 16);
  }
  *(u32x4*)&Bp[t * 8] = u32x4{w[0], w[1], w[2], w[3]};
}

// The same for one-byte elements: 8 bytes per lane, 512-byte runs.
__global__ __launch_bounds__(256) void pack_b8(const uint8_t* __restrict__ B, uint8_t* __restrict__ Bp, int64_t K,
                                               int64_t N, int64_t runs) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= runs * 64) return;
  const int64_t run = t / 64, KB = (K + 31) / 32;
  const int l = (int)(t % 64);
  const int64_t p = run / KB, f = run % KB;
  const int64_t n = p * 16 + (l & 15), k0 = f * 32 + 8 * (l >> 4);
  uint32_t w[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    uint32_t v = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int64_t k = k0 + 4 * h + e;
      v |= (uint32_t)((n < N && k < K) ? B[k * N + n] : 0) << (8 * e);
    }
    w[h] = v;
  }
  *(u32x2*)&Bp[t * 8] = u32x2{w[0], w[1]};
}

hipError_t launch_pack_b8(const uint8_t* B, uint8_t* Bp, int64_t K, int64_t N, hipStream_t st) {
  const int64_t runs = ((N + 15) / 16) * ((K + 31) / 32);
  const int64_t blocks = (runs * 64 + 255) / 256;
  if (blocks == 0) return hipSuccess;
  hipLaunchKernelGGL(pack_b8, dim3((unsigned)blocks), dim3(256), 0, st, B, Bp, K, N, runs);
  return hipGetLastError();
}

hipError_t launch_pack_b(const uint16_t* B, uint16_t* Bp, int64_t K, int64_t N, hipStream_t st) {
  const int64_t runs = ((N + 15) / 16) * ((K + 31) / 32);
  const int64_t blocks = (runs * 64 + 255) / 256;
  if (blocks == 0) return hipSuccess;
  hipLaunchKernelGGL(pack_b, dim3((unsigned)blocks), dim3(256), 0, st, B, Bp, K, N, runs);
  return hipGetLastError();
}

template <int TMS, int D, bool AVEC>
static hipError_t launch_panel_t(const GemmArgs& a, hipStream_t st) {
  dim3 grid((unsigned)((a.N + 15) / 16), (unsigned)((a.M + 16 * TMS - 1) / (16 * TMS)), (unsigned)a.S);
  const bool strided = a.split_w != 0;
  const int bt = a.b_e4m3 ? 2 : a.in_f16 ? 1 : 0;
  auto go = [&](auto BT_) {
    constexpr int BT = decltype(BT_)::value;
    if (strided) hipLaunchKernelGGL((gemm_panel<TMS, D, AVEC, true, BT>), grid, dim3(64), 0, st, a);
    else hipLaunchKernelGGL((gemm_panel<TMS, D, AVEC, false, BT>), grid, dim3(64), 0, st, a);
  };
  if (bt == 2) go(std::integral_constant<int, 2>{});
  else if (bt == 1) go(std::integral_constant<int, 1>{});
  else go(std::integral_constant<int, 0>{});
  return hipGetLastError();
}

// (rows of A per wave / 16, ring depth) pairs built, for 16-byte A runs and
// for element loads
#define DG_PANEL_LIST(X) \
  X(1, 8) X(1, 16) X(1, 24) X(1, 32) X(2, 8) X(2, 12) X(2, 16) X(4, 6) X(4, 10)
#define DG_PANEL_ELEM_LIST(X) X(1, 4) X(2, 2) X(4, 1)

// Ring depths measured best on MI355X (4096 x 4096 B, M = 1, 7, 32, 64)
int panel_default_depth(int tms, bool avec) {
  if (!avec) return tms == 1 ? 4 : tms == 2 ? 2 : 1;
  return tms == 1 ? 16 : tms == 2 ? 16 : 10;
}

bool panel_supported(int tms, int depth, bool avec) {
#define DG_PANEL_HAS(T_, D_) \
  if (tms == T_ && depth == D_) return true;
  if (avec) {
    DG_PANEL_LIST(DG_PANEL_HAS)
  } else {
    DG_PANEL_ELEM_LIST(DG_PANEL_HAS)
  }
#undef DG_PANEL_HAS
  return false;
}

hipError_t launch_gemm_panel(const GemmArgs& a, int tms, int depth, bool avec, hipStream_t st) {
#define DG_PANEL_RUN(T_, D_) \
  if (tms == T_ && depth == D_) return launch_panel_t<T_, D_, AVEC_>(a, st);
  if (avec) {
    constexpr bool AVEC_ = true;
    DG_PANEL_LIST(DG_PANEL_RUN)
  } else {
    constexpr bool AVEC_ = false;
    DG_PANEL_ELEM_LIST(DG_PANEL_RUN)
  }
#undef DG_PANEL_RUN
  return hipErrorInvalidValue;
}

}  // namespace dg
