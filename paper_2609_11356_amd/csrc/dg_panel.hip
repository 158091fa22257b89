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
// An e4m3 B (one byte per element) packs two k blocks per 1 KB run: lane
// l's 16 bytes are its 8 k of the first block, then its 8 k of the second,
// so each load still moves 1 KB (a 512-byte run per block measured slower
// than bf16 at one row: the loads, not the bytes, set the pace) and e4m3
// parts start on 64-k runs.  The wave widens each block's 8 values to bf16
// with the part's conversion instruction (exact) just before the bf16
// instruction, so the order and bits are those of the bf16 GEMM on the
// widened B, with half the bytes streamed.
#include <type_traits>

#include "dg_device.h"
#include "dg_internal.h"
#include "dg_mma.h"

namespace dg {

namespace {

constexpr uint32_t kOOB = 0x80000000u;   // a buffer offset past any record: reads zero

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
// (1 KB runs of two blocks, widened to bf16 before the instruction).  The
// ring holds D runs (BPR blocks each) with the A fragments of their blocks.
template <int TMS, int D, bool AVEC, bool STRIDED, int BT>
__global__ __launch_bounds__(64) void gemm_panel(GemmArgs a) {
  constexpr bool F16 = BT == 1;
  constexpr int BPR = BT == 2 ? 2 : 1;         // k blocks per 1 KB run
  constexpr int RUN = 1024;
  static_assert(!AVEC || (D - 1) * (1 + BPR * TMS) <= 63, "the ring's waits fit the load counter");
  const int lane = threadIdx.x;
  const int64_t panel = blockIdx.x;
  const int64_t i0 = (int64_t)blockIdx.y * 16 * TMS, j0 = panel * 16;
  const int s = blockIdx.z;
  // every k block index and byte offset fits 31 bits (the host keeps the
  // packed B under 2 GiB and A's rows under 2 GiB)
  const int KR = (int)((a.K + 32 * BPR - 1) / (32 * BPR)), K = (int)a.K;
  // blocks (nf) and runs (nr) of part s: contiguous from run r0 (the host
  // puts interior cuts on run boundaries), or dealt tiles of 2^lgw blocks
  // (2^lgr runs)
  int nf = 0, r0 = 0, lgr = 0;
  if constexpr (STRIDED) {
    const int lgw = __builtin_ctz((unsigned)(a.split_w / 32));
    lgr = lgw - (BPR == 2 ? 1 : 0);
    const int w = (int)a.split_w, ntile = (K + w - 1) / w;
    nf = ntile > s ? ((ntile - s + a.S - 1) / a.S) << lgw : 0;
  } else if (a.cuts[s + 1] > a.cuts[s]) {
    r0 = (int)(a.cuts[s] / (32 * BPR));
    nf = (int)((a.cuts[s + 1] + 31) / 32) - BPR * r0;
  }
  const int nr = (nf + BPR - 1) / BPR;
  const int64_t recA = (a.M - i0) * a.K * 2, recB = ((a.N + 15) / 16) * (int64_t)KR * RUN;
  const __amdgpu_buffer_rsrc_t rA = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a.A + i0 * a.K), (short)0, (int)(recA < 0x7fffffff ? recA : 0x7fffffff), 0x00020000);
  // the panel's runs: a base moved to the panel, the run in the scalar offset
  const __amdgpu_buffer_rsrc_t rB = __builtin_amdgcn_make_buffer_rsrc((void*)a.B, (short)0, (int)recB, 0x00020000);
  const int kl = 8 * (lane >> 4);   // the lane's first k within a block
  // lane constants: B's run slot; A's row run (out of range past M), and the
  // first block whose 8 k of this lane lie at or past K (only the last block
  // when K % 32 != 0).  A block's offset goes in the scalar buffer offset.
  const uint32_t vb = (uint32_t)(panel * KR * RUN) + (uint32_t)lane * 16;
  const int flim = (K - kl + 31) / 32;
  uint32_t va[TMS];
#pragma unroll
  for (int mi = 0; mi < TMS; ++mi) {
    const int row = 16 * mi + (lane & 15);
    va[mi] = (i0 + row < a.M) ? (uint32_t)((row * K + kl) * 2) : kOOB;
  }
  // runs g < nre are real (a strided part's last dealt tile may run past
  // K's last run: those runs read as zeros)
  const int nre = STRIDED ? nr : (nr < KR - r0 ? nr : KR - r0);

  // run g of the part -> global run
  auto run_of = [&](int g) -> int {
    if constexpr (STRIDED) return ((s + a.S * (g >> lgr)) << lgr) + (g & ((1 << lgr) - 1));
    else return r0 + g;
  };
  // the ring: one run of B (16 bytes per lane) and the A fragments of its blocks
  u32x4 rb[D];
  u32x4 ra[D][BPR][TMS];
  auto load = [&](int u, int g) {
    const int R = run_of(g);
    const bool ok = g < nre && (!STRIDED || R < KR);
    const int so = ok ? R : 0;
    rb[u] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rB, ok ? vb : kOOB, so * RUN, 0));
#pragma unroll
    for (int h = 0; h < BPR; ++h) {
      const int f = BPR * so + h;
#pragma unroll
      for (int mi = 0; mi < TMS; ++mi) {
        if constexpr (AVEC) {
          ra[u][h][mi] = __builtin_bit_cast(
              u32x4, __builtin_amdgcn_raw_buffer_load_b128(rA, (ok && f < flim) ? va[mi] : kOOB, f * 64, 0));
        } else {
          const int row = 16 * mi + (lane & 15);
          ra[u][h][mi] = load_a_elems(rA, (int64_t)row * a.K, (int64_t)f * 32 + kl, a.K, ok && i0 + row < a.M);
        }
      }
    }
  };

  floatx4 acc[TMS];
#pragma unroll
  for (int mi = 0; mi < TMS; ++mi) acc[mi] = floatx4{0.f, 0.f, 0.f, 0.f};
  // The loads stay in ring order (no scheduling across the barriers): the
  // waits count on run g's loads being older than those of g + 1.
  static_for<0, D>([&](auto u) {
    load(u, u);
    __builtin_amdgcn_sched_barrier(0);
  });
  for (int base = 0; base < nr; base += D) {
    static_for<0, D>([&](auto u) {
      const int g = base + u;
      // this run's loads are the oldest of D groups in flight
      if constexpr (AVEC) __builtin_amdgcn_s_waitcnt(vmcnt_only((D - 1) * (1 + BPR * TMS)));
#pragma unroll
      for (int h = 0; h < BPR; ++h) {
        if (BPR * g + h < nf) {
          u32x4 bw;
          if constexpr (BT == 2)
            bw = u32x4{e4m3x2_bf16x2<false>(rb[u][2 * h]), e4m3x2_bf16x2<true>(rb[u][2 * h]),
                       e4m3x2_bf16x2<false>(rb[u][2 * h + 1]), e4m3x2_bf16x2<true>(rb[u][2 * h + 1])};
          else
            bw = rb[u];
#pragma unroll
          for (int mi = 0; mi < TMS; ++mi)
            acc[mi] = mfma16t<F16>(__builtin_bit_cast(shortx8, ra[u][h][mi]), __builtin_bit_cast(shortx8, bw),
                                   acc[mi]);
        }
      }
      load(u, g + D);
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

// One-byte elements: every 64 x 16 block (two k blocks) is one 1 KB run, lane
// l's 16 bytes holding its 8 k of the first block, then its 8 k of the
// second: thread t writes lane l = t % 64 of run t / 64 (panel p = run / KR,
// run r = run % KR of the panel).
__global__ __launch_bounds__(256) void pack_b8(const uint8_t* __restrict__ B, uint8_t* __restrict__ Bp, int64_t K,
                                               int64_t N, int64_t runs) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= runs * 64) return;
  const int64_t run = t / 64, KR = (K + 63) / 64;
  const int l = (int)(t % 64);
  const int64_t p = run / KR, r = run % KR;
  const int64_t n = p * 16 + (l & 15), k0 = r * 64 + 8 * (l >> 4);
  uint32_t w[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    uint32_t v = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int64_t k = k0 + 32 * (q >> 1) + 4 * (q & 1) + e;
      v |= (uint32_t)((n < N && k < K) ? B[k * N + n] : 0) << (8 * e);
    }
    w[q] = v;
  }
  *(u32x4*)&Bp[t * 16] = u32x4{w[0], w[1], w[2], w[3]};
}

hipError_t launch_pack_b8(const uint8_t* B, uint8_t* Bp, int64_t K, int64_t N, hipStream_t st) {
  const int64_t runs = ((N + 15) / 16) * ((K + 63) / 64);
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

// an e4m3 ring of D runs holds 2 D TMS A fragments (16 bytes per lane each),
// and its waits count up to (D - 1)(1 + 2 TMS) loads (the counter holds 63)
constexpr bool panel_b8_fits(int tms, int d) { return 2 * d * tms <= 48 && (d - 1) * (1 + 2 * tms) <= 63; }

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
  if (bt == 2) {
    // two blocks per run: the rings whose A fragments fit the registers
    if constexpr (panel_b8_fits(TMS, D)) go(std::integral_constant<int, 2>{});
    else return hipErrorInvalidValue;
  }
  else if (bt == 1) go(std::integral_constant<int, 1>{});
  else go(std::integral_constant<int, 0>{});
  return hipGetLastError();
}

// (rows of A per wave / 16, ring depth) pairs built, for 16-byte A runs and
// for element loads
#define DG_PANEL_LIST(X) \
  X(1, 8) X(1, 16) X(1, 24) X(1, 32) X(2, 8) X(2, 12) X(2, 16) X(4, 6) X(4, 10)
#define DG_PANEL_ELEM_LIST(X) X(1, 4) X(2, 2) X(4, 1)

// Ring depths measured best on MI355X (4096 x 4096 B, M = 1, 7, 32, 64);
// an e4m3 ring's runs hold two blocks each
int panel_default_depth(int tms, bool avec, bool b8) {
  if (!avec) return tms == 1 ? 4 : tms == 2 ? 2 : 1;
  if (b8) return tms == 1 ? 8 : tms == 2 ? 8 : 6;
  return tms == 1 ? 16 : tms == 2 ? 16 : 10;
}

bool panel_supported(int tms, int depth, bool avec, bool b8) {
  if (b8 && !panel_b8_fits(tms, depth)) return false;
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
