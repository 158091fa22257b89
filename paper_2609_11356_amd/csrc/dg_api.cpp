// dg_api.cpp -- host side of libdg: descriptor validation and plan, kernel
// selection (speed only, never order), split-K workspace, error mapping.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <new>
#include <string>
#include <utility>

#include "dg_internal.h"

namespace {

bool in(int v, int lo, int hi) { return v >= lo && v <= hi; }

// Cut points of the split for K (Sec. 3.2.2: contiguous parts, each started
// at zero).  Explicit cuts must lie strictly inside (0, K) and increase.
// Without them the span is ceil(K / S) rounded up to whole tiles and the last
// part takes the rest; a part left empty is a shape error.
dg_status plan_cuts(const dg_desc* d, int64_t K, int64_t* cuts) {
  const int S = d->p.split_k;
  cuts[0] = 0;
  cuts[S] = K;
  if (S == 1) return K >= 0 ? DG_OK : DG_ERR_SHAPE;
  if (d->p.n_cuts) {
    for (int s = 1; s < S; ++s) cuts[s] = d->cuts[s - 1];
  } else {
    int64_t span = (K + S - 1) / S;
    span = (span + d->p.tile_k - 1) / d->p.tile_k * d->p.tile_k;
    for (int s = 1; s < S; ++s) cuts[s] = (int64_t)s * span;
  }
  for (int s = 0; s < S; ++s)
    if (!(cuts[s] < cuts[s + 1])) return DG_ERR_SHAPE;
  return DG_OK;
}

// Canonical text of the descriptor's order.  Every field that can change a
// bit appears in full (all explicit cuts included), so equal texts mean equal
// descriptors up to fields that cannot change bits.  Returns false if the text
// does not fit d->sig (it always fits: 63 cuts of at most 20 characters and
// the fixed fields stay far below its size), and create then refuses.
bool make_signature(dg_desc* d) {
  const dg_desc_params& p = d->p;
  // fma = 1 folds the same 8-k chunks whatever the instruction's K
  // on the scalar path a bf16 product is exact, so fma cannot change bits
  // (likewise the same 16-k chunks for the fp8 instructions)
  const bool scalar = p.mma == DG_MMA_SCALAR_FMA;
  const bool f8 = p.in_dtype == DG_IN_E4M3;
  std::string grp = scalar ? "scalar-fma" : p.fma ? (f8 ? "chunk16" : "chunk8") : "group" + std::to_string(d->group);
  char base[512];
  int n = std::snprintf(base, sizeof base,
                        "gfx950-%s-%s/%s/fma%d/tile%d/%s/S%d/%s/merge-%s/partial-%s/merge-dt-%s/"
                        "out-%s/epi%d/%s/leaf%d/%s",
                        f8 ? "e4m3" : "bf16", scalar ? "fma" : "mfma", grp.c_str(), scalar ? 1 : p.fma, p.tile_k,
                        p.tile_combine == DG_CARRY ? "carry" : p.tile_combine == DG_SEQ ? "seq" : "tree",
                        p.split_k, p.tail == DG_TAIL_FIRST ? "tail-first" : "tail-last",
                        p.split_combine == DG_SEQ ? "seq" : "tree", p.partial_dtype ? "bf16" : "f32",
                        p.merge_dtype ? "bf16" : "f32", p.out_dtype ? "bf16" : "f32", p.epilogue,
                        p.epi_round ? "pre-act" : "final", p.leaf_w, p.reduce_op ? "sumsq" : "sum");
  if (n <= 0 || n >= (int)sizeof base) return false;
  std::string s(base);
  // the row reduction's leaf layout and lane fold, when not the defaults (one
  // lane has nothing to fold)
  if (p.leaf_layout == DG_LEAF_STRIDED)
    s += std::string("/leaf-strided") + (p.lane_fold == DG_FOLD_DOWN && p.leaf_w > 1 ? "/fold-down" : "");
  if (p.norm_round == DG_NORM_PRE_WEIGHT) s += "/norm-pre-weight";
  if (p.in_dtype == DG_IN_F16) s += "/in-f16";
  if (p.in_dtype == DG_IN_BF16_E4M3) s += "/in-bf16xe4m3";
  // one strided part is the whole axis, as one contiguous part is
  if (p.split_layout == DG_SPLIT_STRIDED && p.split_k > 1) s += "/strided:" + std::to_string(p.split_tile);
  if (p.n_cuts) {
    s += "/cuts";
    for (int i = 0; i < p.n_cuts; ++i) s += ":" + std::to_string((long long)d->cuts[i]);
  }
  if (s.size() + 1 > sizeof d->sig) return false;
  std::memcpy(d->sig, s.c_str(), s.size() + 1);
  return true;
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

// Block width of the fp8 kernel's 256-row blocks (speed only): 256 x 128 blocks
// run two per CU, so one block's prologue and epilogue overlap the other's
// main loop (MLP 2048 x 14336 x 4096 with bias + SiLU: 148 against 172 us)
constexpr int F8_AUTO_TN = 128;

// ------------------------------------------------------------ workspace

struct Workspace {
  void* ptr = nullptr;
  size_t bytes = 0;
};
std::mutex g_ws_mutex;
std::map<std::pair<int, hipStream_t>, Workspace> g_ws;

// Workspace of at least `bytes` owned by (current device, stream).  Growth is
// stream-ordered (hipMallocAsync / hipFreeAsync on that stream), so launches
// already enqueued on the stream keep their buffer until they finish.
dg_status get_workspace(hipStream_t st, size_t bytes, void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return DG_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_ws_mutex);
  Workspace& w = g_ws[{dev, st}];
  if (w.bytes < bytes) {
    size_t want = bytes + bytes / 4;
    void* p = nullptr;
    if (hipMallocAsync(&p, want, st) != hipSuccess) {
      (void)hipGetLastError();
      return DG_ERR_NOMEM;
    }
    if (w.ptr) (void)hipFreeAsync(w.ptr, st);
    w.ptr = p;
    w.bytes = want;
  }
  *out = w.ptr;
  return DG_OK;
}

// Tile shape for the tiled kernel: a speed choice only.
// The library's choice of kernel and tiles for the chunk-grid kernels
// (speed only; every choice gives the same bits).  Measured on MI355X at
// N = K = 4096 and at the decode and MLP shapes: few rows stream B through
// the deep-ring kernel (whole 128-byte B rows per workgroup once the grid
// is wide enough); larger M goes to the ping-pong kernel with 256 x 256
// blocks when they fill most of the chip (mixed with 256 x 192 blocks when
// that makes the last round over the chip fuller), else with 128 x 128
// blocks, and
// to the transposing-read kernel (two workgroups per CU, XCD-contiguous
// grouped order) when even those are too few.
struct AutoConfig {
  int kern, tm, tn, order, occ, depth, slab_k;
};

// The ping-pong kernels address their operands with 31-bit byte offsets from
// the block's first A row and the part's first B row.
bool pp_fits(const dg::GemmArgs& a) {
  const int64_t lim = 0x7fffffff;
  if (256 * a.K * 2 + 64 > lim || 66 * a.N * 2 > lim) return false;
  for (int s = 0; s < a.S; ++s)
    if ((a.cuts[s + 1] - a.cuts[s] + 4 * 64) * a.N * 2 > lim) return false;
  return true;
}

// Compute units of the current device (cached per device; 256 on MI355X).
int cu_count() {
  static int cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (!cached[dev]) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

// Columns for 256-wide blocks in the mixed-width ping-pong launch, or -1
// when 256-wide blocks alone are as good.  One block runs per CU; the
// estimate counts rounds of blocks over the chip, a 192-wide block taking
// 7/8 of the time of a 256-wide one (measured on MI355X: 117 us for 256
// blocks of 256 x 192 against 131 us for 256 of 256 x 256 at K = 4096;
// the A side of the block's LDS and load traffic does not shrink).
int64_t mixed_split(int64_t M, int64_t N, int S, int ncu) {
  const int64_t tm = S * ((M + 255) / 256);
  auto rounds = [&](int64_t blocks) { return (double)((blocks + ncu - 1) / ncu); };
  const double plain = rounds(tm * ((N + 255) / 256));
  double best = 0.97 * plain;
  int64_t split = -1;
  for (int64_t c = 0; 256 * c <= N; ++c) {
    const double est = rounds(tm * c) + 0.875 * rounds(tm * ((N - 256 * c + 191) / 192));
    if (est < best) {
      best = est;
      split = 256 * c;
    }
  }
  return split;
}

AutoConfig auto_config(int64_t M, int64_t N, int S) {
  if (M <= 32) {
    if (S * ((N + 63) / 64) >= 256) return {4, 16, 64, 0, 0, 4, 64};
    return {4, 16, M <= 16 ? 16 : 32, 0, 0, 2, 256};
  }
  if (M <= 128) return {4, 32, 64, 0, 0, 2, 256};
  const int64_t tiles256 = S * ((M + 255) / 256) * ((N + 255) / 256);
  const int64_t tiles128 = S * ((M + 127) / 128) * ((N + 127) / 128);
  // 256 x 256 blocks, each XCD given a contiguous range of them (2-3 % over
  // row-major order at 4096 x 4096 x 4096 on MI355X)
  if (tiles256 >= 192) return {5, 256, 256, 3, 0, 0, 0};
  if (tiles128 >= 128) return {5, 128, 128, 3, 0, 0, 0};
  return {3, 64, 128, 3, 2, 0, 0};
}

}  // namespace

extern "C" {

int32_t dg_version(void) { return 600; }

const char* dg_strerror(dg_status s) {
  switch (s) {
    case DG_OK: return "ok";
    case DG_ERR_INVALID: return "invalid argument";
    case DG_ERR_UNSUPPORTED: return "unsupported descriptor or knob";
    case DG_ERR_SHAPE: return "shape inconsistent with the descriptor's plan";
    case DG_ERR_ALIGN: return "misaligned pointer";
    case DG_ERR_NOMEM: return "workspace allocation failed";
    case DG_ERR_HIP: return "HIP runtime error";
    case DG_ERR_SCRATCH: return "split-K partials exceed the fixed scratch of the no-allocation entry point";
  }
  return "unknown status";
}

dg_status dg_desc_create(const dg_desc_params* p, dg_desc** out) {
  if (!p || !out) return DG_ERR_INVALID;
  *out = nullptr;
  if (p->struct_size < sizeof(dg_desc_params)) return DG_ERR_INVALID;
  int group;
  if (p->mma == DG_MMA_16X16X32_BF16 || p->mma == DG_MMA_16X16X32_FP8) group = 32;
  else if (p->mma == DG_MMA_32X32X16_BF16 || p->mma == DG_MMA_32X32X16_FP8) group = 16;
  else if (p->mma == DG_MMA_16X16X128_F8F6F4) group = 128;
  else if (p->mma == DG_MMA_32X32X64_F8F6F4) group = 64;
  else if (p->mma == DG_MMA_SCALAR_FMA) group = 1;
  else return DG_ERR_INVALID;
  if (p->tile_k < group || p->tile_k % group != 0 || p->tile_k > (1 << 30)) return DG_ERR_INVALID;
  if (!in(p->split_k, 1, DG_MAX_SPLIT)) return DG_ERR_INVALID;
  if (p->n_cuts != 0 && p->n_cuts != p->split_k - 1) return DG_ERR_INVALID;
  if (p->n_cuts && !p->k_cuts) return DG_ERR_INVALID;
  for (int i = 0; i < p->n_cuts; ++i)
    if (p->k_cuts[i] <= 0 || (i && p->k_cuts[i] <= p->k_cuts[i - 1])) return DG_ERR_INVALID;
  if (!in(p->tile_combine, DG_CARRY, DG_TREE)) return DG_ERR_INVALID;
  if (p->split_combine != DG_SEQ && p->split_combine != DG_TREE) return DG_ERR_INVALID;
  if (!in(p->tail, DG_TAIL_LAST, DG_TAIL_FIRST) || !in(p->fma, 0, 1)) return DG_ERR_INVALID;
  if (!in(p->partial_dtype, DG_F32, DG_BF16) || !in(p->merge_dtype, DG_F32, DG_BF16) ||
      !in(p->out_dtype, DG_F32, DG_BF16))
    return DG_ERR_INVALID;
  if (!in(p->epilogue, DG_EPI_NONE, DG_EPI_BIAS_SILU) || !in(p->epi_round, DG_ROUND_FINAL, DG_ROUND_PRE_ACT))
    return DG_ERR_INVALID;
  if (p->leaf_w < 1 || !in(p->reduce_op, DG_OP_SUM, DG_OP_SUMSQ)) return DG_ERR_INVALID;
  if (!in(p->split_layout, DG_SPLIT_CONTIGUOUS, DG_SPLIT_STRIDED)) return DG_ERR_INVALID;
  if (!in(p->leaf_layout, DG_LEAF_CONTIGUOUS, DG_LEAF_STRIDED) || !in(p->lane_fold, DG_FOLD_UP, DG_FOLD_DOWN))
    return DG_ERR_INVALID;
  if (!in(p->norm_round, DG_NORM_FINAL, DG_NORM_PRE_WEIGHT)) return DG_ERR_INVALID;
  if (!in(p->in_dtype, DG_IN_BF16, DG_IN_E4M3)) return DG_ERR_INVALID;
  // e4m3 x e4m3 goes with an fp8 instruction, and an fp8 instruction with it
  if ((p->in_dtype == DG_IN_E4M3) != in(p->mma, DG_MMA_16X16X32_FP8, DG_MMA_32X32X64_F8F6F4)) return DG_ERR_INVALID;
  if (p->in_dtype == DG_IN_BF16_E4M3 && p->mma == DG_MMA_SCALAR_FMA) return DG_ERR_UNSUPPORTED;
  if (p->split_layout == DG_SPLIT_STRIDED) {
    if (p->split_tile < p->tile_k || p->split_tile % p->tile_k != 0 || p->split_tile > (1 << 30))
      return DG_ERR_INVALID;
    if (p->n_cuts != 0 || p->tail != DG_TAIL_LAST) return DG_ERR_INVALID;
  } else if (p->split_tile != 0) {
    return DG_ERR_INVALID;
  }
  if (p->merge_dtype == DG_BF16 && p->partial_dtype != DG_BF16) return DG_ERR_UNSUPPORTED;
  if (p->epi_round == DG_ROUND_PRE_ACT && p->epilogue != DG_EPI_BIAS_SILU) return DG_ERR_UNSUPPORTED;
  // strided leaves: up to 256 lanes, a power of two; the count-down fold only
  // over strided lanes
  if (p->leaf_layout == DG_LEAF_STRIDED && (p->leaf_w > 256 || (p->leaf_w & (p->leaf_w - 1))))
    return DG_ERR_UNSUPPORTED;
  if (p->lane_fold == DG_FOLD_DOWN && p->leaf_layout != DG_LEAF_STRIDED) return DG_ERR_UNSUPPORTED;
  dg_desc* d = new (std::nothrow) dg_desc;
  if (!d) return DG_ERR_NOMEM;
  std::memset(d, 0, sizeof *d);
  d->p = *p;
  d->p.struct_size = sizeof(dg_desc_params);
  for (int i = 0; i < p->n_cuts; ++i) d->cuts[i] = p->k_cuts[i];
  d->p.k_cuts = p->n_cuts ? d->cuts : nullptr;
  d->group = group;
  if (!make_signature(d)) {
    delete d;
    return DG_ERR_UNSUPPORTED;
  }
  *out = d;
  return DG_OK;
}

void dg_desc_destroy(dg_desc* d) { delete d; }

dg_status dg_desc_signature(const dg_desc* d, char* buf, size_t n) {
  if (!d || !buf) return DG_ERR_INVALID;
  size_t len = std::strlen(d->sig);
  if (n < len + 1) return DG_ERR_INVALID;
  std::memcpy(buf, d->sig, len + 1);
  return DG_OK;
}

// The GEMM; with colsum_part set, a launch on 256-row blocks of one part
// also writes the column sums of each 256-row run of C there, and *fused says
// whether it did.
static dg_status gemm_impl(const dg_desc* d, const void* A, const void* B, const void* bias, void* C,
                           int64_t M, int64_t N, int64_t K, const dg_knobs* knobs, void* stream,
                           float* colsum_part, bool* fused, bool noalloc = false, bool packed = false) {
  if (fused) *fused = false;
  if (!d) return DG_ERR_INVALID;
  if (M < 0 || N < 0 || K < 0) return DG_ERR_SHAPE;
  const dg_desc_params& p = d->p;
  const bool need_bias = p.epilogue != DG_EPI_NONE;
  int kern = knobs ? knobs->kernel : 0;
  int tm = knobs ? knobs->tile_m : 0, tn = knobs ? knobs->tile_n : 0;
  int order = knobs ? knobs->order : 0, occ = knobs ? knobs->occupancy : 0;
  int depth = knobs ? knobs->depth : 0, slab_k = knobs ? knobs->slab_k : 0;
  int64_t split_n = knobs ? knobs->split_n : 0;
  if (!in(kern, 0, 14) || !in(order, 0, 3) || !in(occ, 0, 2)) return DG_ERR_UNSUPPORTED;
  // packed B runs on kernel 11 only, and kernel 11 runs nothing else
  if (packed ? (kern != 0 && kern != 11) : kern == 11) return DG_ERR_UNSUPPORTED;
  if (packed) kern = 11;
  // the scalar instruction runs on kernel 9 only, and kernel 9 runs nothing else
  const bool scalar = p.mma == DG_MMA_SCALAR_FMA;
  if (scalar ? (kern != 0 && kern != 9) : kern == 9) return DG_ERR_UNSUPPORTED;
  if (kern == 9 && (tm || tn || order || occ || depth || slab_k || split_n)) return DG_ERR_UNSUPPORTED;
  // binary16 operands: the generic, v3, few-row, ping-pong and scalar kernels
  const bool f16 = p.in_dtype == DG_IN_F16;
  if (f16 && (kern == 2 || kern == 7 || kern == 8 || kern == 10)) return DG_ERR_UNSUPPORTED;
  // an e4m3 B: the generic kernel (row-major) and the packed kernel only
  const bool b8 = p.in_dtype == DG_IN_BF16_E4M3;
  if (b8 && !packed && kern == 0) kern = 1;
  if (b8 && kern != 1 && kern != 11) return DG_ERR_UNSUPPORTED;
  // e4m3 x e4m3: the generic kernel (any descriptor) or the fp8 tiled kernel
  // 13 (a carried accumulator); kernel 13 runs nothing else and takes no knob
  const bool f8 = p.in_dtype == DG_IN_E4M3;
  if (f8 && (packed || !(kern == 0 || kern == 1 || kern == 13))) return DG_ERR_UNSUPPORTED;
  if (!f8 && kern == 13) return DG_ERR_UNSUPPORTED;
  // kernel 14: bf16 operands only, no knob
  if (kern == 14 && (p.in_dtype != DG_IN_BF16 || tm || tn || order || occ || depth || slab_k || split_n))
    return DG_ERR_UNSUPPORTED;
  // kernel 13 blocks: 128 x 128, 256 x 256 or 256 x 128 (tile_m, tile_n)
  if (kern == 13 && (order || occ || depth || slab_k || split_n ||
                     !((tm == 0 && tn == 0) || (tm == 128 && (tn == 0 || tn == 128)) ||
                       (tm == 256 && (tn == 0 || tn == 128 || tn == 256)))))
    return DG_ERR_UNSUPPORTED;
  if (kern != 3 && kern != 5 && kern != 6 && kern != 7 && kern != 10 && order) return DG_ERR_UNSUPPORTED;
  if ((kern == 6 || kern == 7 || kern == 10) && (tm || tn || split_n < 0 || split_n % 256 || split_n > N))
    return DG_ERR_UNSUPPORTED;
  if (kern != 6 && kern != 7 && kern != 10 && split_n) return DG_ERR_UNSUPPORTED;
  if (kern != 3 && occ) return DG_ERR_UNSUPPORTED;
  if (kern == 5 && (tm || tn) && !dg::wide_supported(tm, tn)) return DG_ERR_UNSUPPORTED;
  if (kern != 4 && kern != 8 && kern != 11 && (depth || slab_k)) return DG_ERR_UNSUPPORTED;
  if (kern == 11 && (slab_k || tn || order || occ || split_n || !(tm == 0 || tm == 16 || tm == 32 || tm == 64)))
    return DG_ERR_UNSUPPORTED;
  if (kern == 4 && !dg::skinny_supported(tm ? tm : 16, tn ? tn : 64, depth, slab_k)) return DG_ERR_UNSUPPORTED;
  if (kern == 8 && !dg::skinny_dma_supported(tm ? tm : 16, tn ? tn : 16, depth ? depth : 8, slab_k ? slab_k : 256))
    return DG_ERR_UNSUPPORTED;
  if (kern == 12 && (tm || tn)) return DG_ERR_UNSUPPORTED;
  if (kern != 4 && kern != 5 && kern != 8 && kern != 11 && kern != 13 && (tm || tn) &&
      !(tm && tn && (kern == 3 ? dg::v3_supported(tm, tn, occ == 2 ? 2 : 1) : dg::tiled_supported(tm, tn))))
    return DG_ERR_UNSUPPORTED;
  // A strided split runs on the generic kernel or on the few-row kernel with
  // one dealt tile per slab.
  if (p.split_layout == DG_SPLIT_STRIDED && p.split_k > 1 && kern != 0 && kern != 1 && kern != 9 && kern != 11 &&
      !((kern == 4 || kern == 8) && slab_k == p.split_tile))
    return DG_ERR_UNSUPPORTED;
  if (M == 0 || N == 0) return DG_OK;
  if (!C || (need_bias && !bias) || (K > 0 && (!A || !B))) return DG_ERR_INVALID;
  if (!aligned(A, f8 ? 1 : 2) || !aligned(B, (b8 || f8) ? 1 : 2) || !aligned(C, p.out_dtype == DG_F32 ? 4 : 2) ||
      (need_bias && !aligned(bias, 2)))
    return DG_ERR_ALIGN;
  if (K == 0 && p.split_k > 1) return DG_ERR_SHAPE;

  dg::GemmArgs a;
  std::memset(&a, 0, sizeof a);
  const bool strided = p.split_layout == DG_SPLIT_STRIDED && p.split_k > 1;
  if (strided) {
    // parts are dealt tiles, not ranges: the kernels read split_w instead
    a.split_w = p.split_tile;
    a.cuts[0] = 0;
    for (int s = 1; s <= p.split_k; ++s) a.cuts[s] = K;
  } else if (K > 0) {
    dg_status st = plan_cuts(d, K, a.cuts);
    if (st != DG_OK) return st;
  } else {
    a.cuts[0] = a.cuts[1] = 0;
  }
  a.A = (const uint16_t*)A;
  a.B = (const uint16_t*)B;
  a.bias = (const uint16_t*)bias;
  a.C = C;
  a.M = M;
  a.N = N;
  a.K = K;
  a.S = p.split_k;
  a.tile_k = p.tile_k;
  a.group = d->group;
  a.tile_combine = p.tile_combine;
  a.tail_first = p.tail == DG_TAIL_FIRST;
  a.fma = p.fma;
  a.partial_bf16 = p.partial_dtype == DG_BF16;
  a.out_bf16 = p.out_dtype == DG_BF16;
  a.epilogue = p.epilogue;
  a.pre_act = p.epi_round == DG_ROUND_PRE_ACT;
  a.in_f16 = f16;
  a.b_e4m3 = b8;
  a.ab_e4m3 = f8;
  if ((M + 15) / 16 > 65535 || (N + 15) / 16 > (int64_t)1 << 31) return DG_ERR_SHAPE;

  // The packed-B kernel (dg_panel.hip): one accumulator carried through the
  // part's 32-k blocks, parts starting on a block, dealt tiles of 2^j blocks.
  int panel_tms = 0, panel_depth = 0;
  bool panel_avec = false;
  if (packed) {
    if (scalar || p.tile_combine != DG_CARRY || p.fma != 1 || p.tail == DG_TAIL_FIRST || M > 64)
      return DG_ERR_UNSUPPORTED;
    // runs of 32 k (bf16, binary16) or 64 k (e4m3): parts start on a run
    const int64_t run_k = b8 ? 64 : 32;
    if (strided) {
      const int64_t wf = p.split_tile / run_k;
      if (p.split_tile % run_k || (wf & (wf - 1))) return DG_ERR_UNSUPPORTED;
    } else {
      for (int s = 1; s < a.S; ++s)
        if (a.cuts[s] % run_k) return DG_ERR_UNSUPPORTED;
    }
    if (!aligned(B, 16)) return DG_ERR_ALIGN;
    // every buffer offset (the packed B, A's rows) stays in 31 bits
    if ((b8 ? dg_packed_b8_bytes(K, N) : dg_packed_b_bytes(K, N)) > 0x7fffffff || M * K * 2 > 0x7fffffff)
      return DG_ERR_UNSUPPORTED;
    panel_tms = tm ? tm / 16 : (M <= 16 ? 1 : M <= 32 ? 2 : 4);
    panel_avec = K % 8 == 0 && aligned(A, 16);
    panel_depth = depth ? depth : dg::panel_default_depth(panel_tms, panel_avec, b8);
    if (!dg::panel_supported(panel_tms, panel_depth, panel_avec, b8)) return DG_ERR_UNSUPPORTED;
  }

  // The fp8 tiled kernel: a carried accumulator with fma = 1 (the 16-k chunk
  // chain), 16-byte rows (K, N multiples of 16) and the chunk grid on
  // multiples of 16 from k = 0 (parts and a leading short tile).
  // (decided before any workspace is taken)
  if (f8) {
    bool f8_ok = p.tile_combine == DG_CARRY && p.fma == 1 && !strided && K % 16 == 0 && N % 16 == 0 &&
                 aligned(A, 16) && aligned(B, 16) && aligned(C, 16) && (!need_bias || aligned(bias, 16));
    for (int s = 0; s < a.S && f8_ok; ++s) {
      const int64_t len = a.cuts[s + 1] - a.cuts[s];
      if (a.cuts[s] % 16 || (a.tail_first && (len % p.tile_k) % 16)) f8_ok = false;
    }
    if (kern == 13 && !f8_ok) return DG_ERR_UNSUPPORTED;
    if (kern == 0) kern = f8_ok ? 13 : 1;
    // 256-row blocks (buffer offsets: M K and K N bytes below 2^31) from
    // 129 rows on, else 128 x 128
    if (kern == 13) {
      const bool big_ok = M * K < 0x7fffffff && K * N < 0x7fffffff;
      if (tm == 256 && !big_ok) return DG_ERR_UNSUPPORTED;
      if (!tm) tm = (M > 128 && big_ok) ? 256 : 128;
      if (!tn) tn = tm == 256 ? F8_AUTO_TN : 128;
    }
  }
  hipStream_t st = (hipStream_t)stream;
  if (a.S > 1) {
    void* ws = nullptr;
    const size_t bytes = (size_t)a.S * (size_t)M * (size_t)N * sizeof(float);
    if (noalloc) {
      // the fixed per-device array; nothing is allocated
      if ((uint64_t)a.S * (uint64_t)M * (uint64_t)N > DG_NOALLOC_SCRATCH_BYTES / sizeof(float))
        return DG_ERR_SCRATCH;
      if (dg::noalloc_scratch(&ws) != hipSuccess) return DG_ERR_HIP;
    } else {
      dg_status s = get_workspace(st, bytes, &ws);
      if (s != DG_OK) return s;
    }
    a.ws = (float*)ws;
  }

  // The tiled kernel needs the chunk grid (8 k from every tile start) to sit
  // on multiples of 8 from k = 0, a carried accumulator, and 16-byte rows.
  bool tiled_ok = !f8 && p.tile_combine == DG_CARRY && p.fma == 1 && K % 8 == 0 && N % 8 == 0 &&
                  aligned(A, 16) && aligned(B, 16) && aligned(C, 16) && (!need_bias || aligned(bias, 16));
  for (int s = 0; s < a.S && tiled_ok; ++s) {
    if (a.cuts[s] % 8) tiled_ok = false;
    int64_t len = a.cuts[s + 1] - a.cuts[s];
    if (a.tail_first && (len % p.tile_k) % 8) tiled_ok = false;
  }
  // The tile-combine kernel (tile chain or tree, or fma = 0, on the tiled
  // layout): the tiled layout's alignment, every tile boundary of every part
  // on a 32-k step from the part start, and for the tree at most 128 tiles
  // per part (its stack lives in registers).
  const bool gen = p.tile_combine != DG_CARRY || p.fma == 0;
  bool tc_ok = gen && !scalar && !strided && !b8 && !f8 && (p.fma == 1 || d->group == 32) && p.tile_k % 32 == 0 &&
               K % 8 == 0 && N % 8 == 0 && aligned(A, 16) && aligned(B, 16) && aligned(C, 16) &&
               (!need_bias || aligned(bias, 16));
  int64_t max_tiles = 0;
  for (int s = 0; s < a.S && tc_ok; ++s) {
    const int64_t len = a.cuts[s + 1] - a.cuts[s];
    if (a.cuts[s] % 8 || (a.tail_first && (len % p.tile_k) % 32)) tc_ok = false;
    max_tiles = std::max<int64_t>(max_tiles, (len + p.tile_k - 1) / p.tile_k);
  }
  int tc_levels = 2;
  while (tc_levels < 7 && max_tiles > ((int64_t)1 << tc_levels)) ++tc_levels;
  if (p.tile_combine == DG_TREE && max_tiles > 128) tc_ok = false;
  if (scalar) {
    tiled_ok = false;
    kern = 9;
  }
  if (kern == 12 && !tc_ok) return DG_ERR_UNSUPPORTED;
  if (kern == 0 && !tiled_ok && tc_ok) kern = 12;
  if (kern >= 2 && kern != 9 && kern != 11 && kern != 12 && kern != 13 && !tiled_ok) return DG_ERR_UNSUPPORTED;
  if (kern == 14 && !(M * K < 0x3fffffff && K * N < 0x3fffffff)) return DG_ERR_UNSUPPORTED;
  if (strided && kern == 0) {
    const int tmc = M <= 16 ? 16 : M <= 32 ? 32 : 64;
    const int tnc = (a.S * ((N + 63) / 64) >= 256) ? 64 : 32;
    if (tiled_ok && M <= 64 && dg::skinny_supported(tmc, tnc, 4, p.split_tile)) {
      kern = 4;
      tm = tmc;
      tn = tnc;
      depth = 4;
      slab_k = p.split_tile;
    } else {
      kern = 1;
    }
  }
  if (kern == 1 && (tm || tn)) return DG_ERR_UNSUPPORTED;
  if (kern == 0 && tiled_ok) {
    AutoConfig c = auto_config(M, N, a.S);
    if (c.kern == 5 && !pp_fits(a)) c = {3, 64, 128, 3, 2, 0, 0};
    if (c.kern == 5 && c.tm == 256 && c.tn == 256) {
      const int64_t sp = mixed_split(M, N, a.S, cu_count());
      if (sp >= 0) {
        // the width mix keeps row-major block order (measured best for it)
        c.kern = 6;
        c.tm = c.tn = 0;
        c.order = 1;
        split_n = sp;
      }
    }
    kern = c.kern;
    tm = c.tm;
    tn = c.tn;
    order = c.order;
    occ = c.occ;
    depth = c.depth;
    slab_k = c.slab_k;
  }
  if (colsum_part && a.S == 1 && (kern == 6 || (kern == 5 && tm == 256))) {
    a.colsum_part = colsum_part;
    *fused = true;
  }
  hipError_t e;
  if (kern == 11) {
    e = dg::launch_gemm_panel(a, panel_tms, panel_depth, panel_avec, st);
  } else if (kern == 14) {
    if (((M + 255) / 256) * ((N + 127) / 128) > INT32_MAX) return DG_ERR_SHAPE;
    a.order = 1;
    e = dg::launch_gemm_b16n(a, st);
  } else if (kern == 13) {
    if (((M + tm - 1) / tm) * ((N + tn - 1) / tn) > INT32_MAX) return DG_ERR_SHAPE;
    a.order = 1;
    e = dg::launch_gemm_f8(a, tm == 256 && tn == 128 ? 256 + 128 : tm, st);
  } else if (kern == 12) {
    if (((M + 127) / 128) * ((N + 63) / 64) > INT32_MAX) return DG_ERR_SHAPE;
    a.order = 1;
    e = dg::launch_gemm_tc(a, tc_levels, st);
  } else if (kern == 9) {
    if ((M + 3) / 4 > 65535 || (N + 255) / 256 > 0x7fffffff) return DG_ERR_SHAPE;
    e = dg::launch_gemm_scalar(a, st);
  } else if (kern == 8) {
    if (!tm) tm = 16;
    if (!tn) tn = 16;
    if (!depth) depth = 8;
    if (!slab_k) slab_k = 256;
    // buffer offsets: a B row run and the slab offset past the part end stay in 31 bits
    const int64_t lim = 0x7fffffff;
    if ((K + (int64_t)(depth + 1) * slab_k * a.S) * N * 2 > lim || (int64_t)tm * K * 2 > lim) return DG_ERR_UNSUPPORTED;
    e = dg::launch_gemm_skinny_dma(a, tm, tn, depth, slab_k, st);
  } else if (kern == 4) {
    e = dg::launch_gemm_skinny(a, tm ? tm : 16, tn ? tn : 64, depth, slab_k, st);
  } else if (kern == 3) {
    if (!tm) { tm = 128; tn = 128; }
    if (((M + tm - 1) / tm) * ((N + tn - 1) / tn) > INT32_MAX) return DG_ERR_SHAPE;
    a.order = order ? order : 1;
    e = dg::launch_gemm_v3(a, tm, tn, occ == 2 ? 2 : 1, st);
  } else if (kern == 5) {
    if (!tm) { tm = 256; tn = 128; }
    if (((M + tm - 1) / tm) * ((N + tn - 1) / tn) > INT32_MAX) return DG_ERR_SHAPE;
    a.order = order ? order : 3;
    if (dg::wide_is_pp(tm, tn) && !pp_fits(a)) return DG_ERR_UNSUPPORTED;
    e = dg::launch_gemm_wide(a, tm, tn, st);
  } else if (kern == 10) {
    if (!pp_fits(a)) return DG_ERR_UNSUPPORTED;
    // split_n 0: the library's split, or 256-wide blocks alone when no split helps
    if (split_n == 0) {
      const int64_t sp = mixed_split(M, N, a.S, cu_count());
      split_n = sp < 0 ? (N + 255) / 256 * 256 : sp;
    }
    if (((M + 255) / 256) * ((split_n + 255) / 256 + (N > split_n ? (N - split_n + 191) / 192 : 0)) > INT32_MAX)
      return DG_ERR_SHAPE;
    a.order = order ? order : 1;
    a.n_split = split_n;
    e = dg::launch_gemm_w4(a, st);
  } else if (kern == 7) {
    if (!pp_fits(a)) return DG_ERR_UNSUPPORTED;
    // split_n 0: the library's split, or 256-wide blocks alone when no split helps
    bool mixed = true;
    if (split_n == 0) {
      const int64_t sp = mixed_split(M, N, a.S, cu_count());
      if (sp < 0) mixed = false;
      else split_n = sp;
    }
    if (((M + 255) / 256) * (split_n / 256 + (N - split_n + 191) / 192 + (N + 255) / 256) > INT32_MAX)
      return DG_ERR_SHAPE;
    a.order = order ? order : 1;
    a.n_split = split_n;
    e = dg::launch_gemm_ppd(a, mixed, st);
  } else if (kern == 6) {
    if (!pp_fits(a)) return DG_ERR_UNSUPPORTED;
    if (knobs && knobs->kernel == 6 && split_n == 0) {
      const int64_t sp = mixed_split(M, N, a.S, cu_count());
      split_n = sp > 0 ? sp : 0;
    }
    if (((M + 255) / 256) * (split_n / 256 + (N - split_n + 191) / 192) > INT32_MAX) return DG_ERR_SHAPE;
    a.order = order ? order : 1;
    a.n_split = split_n;
    e = dg::launch_gemm_pp_mixed(a, st);
  } else if (kern == 2) {
    if (!tm) { tm = 128; tn = 128; }
    if ((M + tm - 1) / tm > 65535) return DG_ERR_SHAPE;
    e = dg::launch_gemm_tiled(a, tm, tn, st);
  } else {
    e = dg::launch_gemm_generic(a, st);
  }
  if (e != hipSuccess) return DG_ERR_HIP;
  if (a.S > 1) {
    dg::CombineArgs c;
    c.ws = a.ws;
    c.bias = a.bias;
    c.C = C;
    c.M = M;
    c.N = N;
    c.S = a.S;
    c.split_combine = p.split_combine;
    c.merge_bf16 = p.merge_dtype == DG_BF16;
    c.out_bf16 = a.out_bf16;
    c.epilogue = a.epilogue;
    c.pre_act = a.pre_act;
    if (dg::launch_splitk_combine(c, st) != hipSuccess) return DG_ERR_HIP;
  }
  return DG_OK;
}

dg_status dg_gemm_knobs(const dg_desc* d, const void* A, const void* B, const void* bias, void* C,
                        int64_t M, int64_t N, int64_t K, const dg_knobs* knobs, void* stream) {
  return gemm_impl(d, A, B, bias, C, M, N, K, knobs, stream, nullptr, nullptr);
}

dg_status dg_gemm(const dg_desc* d, const void* A, const void* B, const void* bias, void* C,
                  int64_t M, int64_t N, int64_t K, void* stream) {
  return dg_gemm_knobs(d, A, B, bias, C, M, N, K, nullptr, stream);
}

dg_status dg_gemm_noalloc(const dg_desc* d, const void* A, const void* B, const void* bias, void* C,
                          int64_t M, int64_t N, int64_t K, void* stream) {
  return gemm_impl(d, A, B, bias, C, M, N, K, nullptr, stream, nullptr, nullptr, true);
}

size_t dg_packed_b_bytes(int64_t K, int64_t N) {
  if (K < 0 || N < 0) return SIZE_MAX;
  const uint64_t panels = (uint64_t)(N + 15) / 16, blocks = (uint64_t)(K + 31) / 32;
  if (panels && blocks > (SIZE_MAX / 1024) / panels) return SIZE_MAX;
  return (size_t)(panels * blocks * 1024);
}

dg_status dg_pack_b(const void* B, void* Bp, int64_t K, int64_t N, void* stream) {
  if (K < 0 || N < 0) return DG_ERR_SHAPE;
  if (K == 0 || N == 0) return DG_OK;
  if (!B || !Bp) return DG_ERR_INVALID;
  if (!aligned(B, 2) || !aligned(Bp, 16)) return DG_ERR_ALIGN;
  if (dg_packed_b_bytes(K, N) == SIZE_MAX || (N + 15) / 16 * ((K + 31) / 32) > ((int64_t)1 << 31) * 4)
    return DG_ERR_SHAPE;
  if (dg::launch_pack_b((const uint16_t*)B, (uint16_t*)Bp, K, N, (hipStream_t)stream) != hipSuccess)
    return DG_ERR_HIP;
  return DG_OK;
}

size_t dg_packed_b8_bytes(int64_t K, int64_t N) {
  if (K < 0 || N < 0) return SIZE_MAX;
  const uint64_t panels = (uint64_t)(N + 15) / 16, runs = (uint64_t)(K + 63) / 64;
  if (panels && runs > (SIZE_MAX / 1024) / panels) return SIZE_MAX;
  return (size_t)(panels * runs * 1024);
}

dg_status dg_pack_b8(const void* B, void* Bp, int64_t K, int64_t N, void* stream) {
  if (K < 0 || N < 0) return DG_ERR_SHAPE;
  if (K == 0 || N == 0) return DG_OK;
  if (!B || !Bp) return DG_ERR_INVALID;
  if (!aligned(Bp, 16)) return DG_ERR_ALIGN;
  if (dg_packed_b8_bytes(K, N) == SIZE_MAX || (N + 15) / 16 * ((K + 63) / 64) > ((int64_t)1 << 31) * 4)
    return DG_ERR_SHAPE;
  if (dg::launch_pack_b8((const uint8_t*)B, (uint8_t*)Bp, K, N, (hipStream_t)stream) != hipSuccess)
    return DG_ERR_HIP;
  return DG_OK;
}

dg_status dg_gemm_packed_knobs(const dg_desc* d, const void* A, const void* Bp, const void* bias, void* C,
                               int64_t M, int64_t N, int64_t K, const dg_knobs* knobs, void* stream) {
  return gemm_impl(d, A, Bp, bias, C, M, N, K, knobs, stream, nullptr, nullptr, false, true);
}

dg_status dg_gemm_packed(const dg_desc* d, const void* A, const void* Bp, const void* bias, void* C,
                         int64_t M, int64_t N, int64_t K, void* stream) {
  return dg_gemm_packed_knobs(d, A, Bp, bias, C, M, N, K, nullptr, stream);
}

dg_status dg_gemm_colsum(const dg_desc* d, const void* A, const void* B, const void* bias, void* C,
                         float* colsum, int64_t M, int64_t N, int64_t K, void* stream) {
  if (!d) return DG_ERR_INVALID;
  if (M < 0 || N < 0 || K < 0) return DG_ERR_SHAPE;
  if (N > 0 && !colsum) return DG_ERR_INVALID;
  if (colsum && !aligned(colsum, 4)) return DG_ERR_ALIGN;
  const int64_t nrun = (M + 255) / 256;
  if (nrun > 65535 || (N + 255) / 256 > 0x7fffffff) return DG_ERR_SHAPE;
  hipStream_t st = (hipStream_t)stream;
  dg::ColsumArgs c;
  c.C = C;
  c.part = nullptr;
  c.colsum = colsum;
  c.M = M;
  c.N = N;
  c.out_bf16 = d->p.out_dtype == DG_BF16;
  // One part: the GEMM's epilogue may fold the 256-row runs itself (run roots
  // straight into colsum when there is one run); the workspace is free then.
  bool fused = false;
  dg_status s;
  if (d->p.split_k == 1 && M > 0 && N > 0) {
    if (nrun > 1) {
      void* ws = nullptr;
      s = get_workspace(st, (size_t)nrun * (size_t)N * sizeof(float), &ws);
      if (s != DG_OK) return s;
      c.part = (float*)ws;
    }
    s = gemm_impl(d, A, B, bias, C, M, N, K, nullptr, stream, nrun > 1 ? c.part : colsum, &fused);
  } else {
    s = dg_gemm_knobs(d, A, B, bias, C, M, N, K, nullptr, stream);
  }
  if (s != DG_OK || N == 0) return s;
  if (fused) {
    if (nrun > 1 && dg::launch_colsum_merge(c, st) != hipSuccess) return DG_ERR_HIP;
    return DG_OK;
  }
  if (nrun > 1 && !c.part) {
    void* ws = nullptr;
    s = get_workspace(st, (size_t)nrun * (size_t)N * sizeof(float), &ws);
    if (s != DG_OK) return s;
    c.part = (float*)ws;
  }
  if (dg::launch_colsum(c, st) != hipSuccess) return DG_ERR_HIP;
  return DG_OK;
}

static dg::RowsumArgs rowsum_args(const dg_desc* d, const float* X, float* out, int64_t rows, int64_t cols) {
  dg::RowsumArgs a;
  std::memset(&a, 0, sizeof a);
  a.X = X;
  a.out = out;
  a.rows = rows;
  a.cols = cols;
  a.leaf_w = d->p.leaf_w;
  a.sumsq = d->p.reduce_op == DG_OP_SUMSQ;
  a.fma = d->p.fma;
  a.strided = d->p.leaf_layout == DG_LEAF_STRIDED;
  a.down = d->p.lane_fold == DG_FOLD_DOWN;
  return a;
}

dg_status dg_rowsum(const dg_desc* d, const float* X, float* out, int64_t rows, int64_t cols,
                    void* stream) {
  if (!d) return DG_ERR_INVALID;
  if (rows < 0 || cols < 0) return DG_ERR_SHAPE;
  if (rows == 0) return DG_OK;
  if (!out || (cols > 0 && !X)) return DG_ERR_INVALID;
  if (!aligned(out, 4) || (X && !aligned(X, 4))) return DG_ERR_ALIGN;
  if ((rows + 3) / 4 > (int64_t)0x7fffffff) return DG_ERR_SHAPE;
  dg::RowsumArgs a = rowsum_args(d, X, out, rows, cols);
  if (dg::launch_rowsum(a, (hipStream_t)stream) != hipSuccess) return DG_ERR_HIP;
  return DG_OK;
}

dg_status dg_softmax(const dg_desc* d, const float* X, void* Y, int64_t rows, int64_t cols, void* stream) {
  if (!d || d->p.reduce_op != DG_OP_SUM) return DG_ERR_INVALID;
  if (rows < 0 || cols < 0) return DG_ERR_SHAPE;
  if (rows == 0 || cols == 0) return DG_OK;
  if (!X || !Y) return DG_ERR_INVALID;
  const bool out_bf16 = d->p.out_dtype == DG_BF16;
  if (!aligned(X, 4) || !aligned(Y, out_bf16 ? 2 : 4)) return DG_ERR_ALIGN;
  if (rows > (int64_t)0x7fffffff) return DG_ERR_SHAPE;
  hipStream_t st = (hipStream_t)stream;
  dg::RowsumArgs a = rowsum_args(d, X, nullptr, rows, cols);
  dg::NormArgs n;
  std::memset(&n, 0, sizeof n);
  n.X = X;
  n.Y = Y;
  n.rows = rows;
  n.cols = cols;
  n.out_bf16 = out_bf16;
  if (dg::softmax_fused_ok(a, n)) {
    if (dg::launch_softmax_fused(a, n, st) != hipSuccess) return DG_ERR_HIP;
    return DG_OK;
  }
  // exponentials to the workspace, their reciprocal sums after them, then the products
  void* ws = nullptr;
  dg_status s = get_workspace(st, (size_t)rows * (size_t)(cols + 1) * sizeof(float), &ws);
  if (s != DG_OK) return s;
  float* E = (float*)ws;
  float* rinv = E + rows * cols;
  dg::NormArgs e = n;
  e.Y = E;
  e.out_bf16 = 0;
  if (dg::launch_softmax_exp(e, st) != hipSuccess) return DG_ERR_HIP;
  a.X = E;
  a.out = rinv;
  a.rms = 2;
  if (dg::launch_rowsum(a, st) != hipSuccess) return DG_ERR_HIP;
  n.X = E;
  n.rinv = rinv;
  if (dg::launch_rmsnorm_scale(n, st) != hipSuccess) return DG_ERR_HIP;
  return DG_OK;
}

dg_status dg_layernorm(const dg_desc* d, const float* X, const void* w, const void* b, float eps, void* Y,
                       int64_t rows, int64_t cols, void* stream) {
  if (!d) return DG_ERR_INVALID;
  if (rows < 0 || cols < 0) return DG_ERR_SHAPE;
  if (rows == 0 || cols == 0) return DG_OK;
  if (!X || !Y) return DG_ERR_INVALID;
  const bool out_bf16 = d->p.out_dtype == DG_BF16;
  if (!aligned(X, 4) || !aligned(Y, out_bf16 ? 2 : 4) || (w && !aligned(w, 2)) || (b && !aligned(b, 2)))
    return DG_ERR_ALIGN;
  if (rows > (int64_t)0x7fffffff) return DG_ERR_SHAPE;
  hipStream_t st = (hipStream_t)stream;
  dg::RowsumArgs a = rowsum_args(d, X, nullptr, rows, cols);
  a.eps = eps;
  dg::NormArgs n;
  std::memset(&n, 0, sizeof n);
  n.X = X;
  n.w = (const uint16_t*)w;
  n.b = (const uint16_t*)b;
  n.Y = Y;
  n.rows = rows;
  n.cols = cols;
  n.out_bf16 = out_bf16;
  n.pre_round = d->p.norm_round == DG_NORM_PRE_WEIGHT;
  if (dg::rmsnorm_fused_ok(a, n)) {
    if (dg::launch_layernorm_fused(a, n, st) != hipSuccess) return DG_ERR_HIP;
    return DG_OK;
  }
  // means, centred values, reciprocal roots, then the scaling
  void* ws = nullptr;
  dg_status s = get_workspace(st, (size_t)rows * (size_t)(cols + 2) * sizeof(float), &ws);
  if (s != DG_OK) return s;
  float* D = (float*)ws;
  float* mean = D + rows * cols;
  float* rinv = mean + rows;
  a.sumsq = 0;
  a.out = mean;
  a.rms = 3;
  if (dg::launch_rowsum(a, st) != hipSuccess) return DG_ERR_HIP;
  dg::NormArgs c = n;
  c.rinv = mean;
  c.Y = D;
  if (dg::launch_layernorm_center(c, st) != hipSuccess) return DG_ERR_HIP;
  a.X = D;
  a.sumsq = 1;
  a.out = rinv;
  a.rms = 1;
  if (dg::launch_rowsum(a, st) != hipSuccess) return DG_ERR_HIP;
  n.X = D;
  n.rinv = rinv;
  if (dg::launch_rmsnorm_scale(n, st) != hipSuccess) return DG_ERR_HIP;
  return DG_OK;
}

dg_status dg_rmsnorm(const dg_desc* d, const float* X, const void* w, float eps, void* Y,
                     int64_t rows, int64_t cols, void* stream) {
  if (!d || d->p.reduce_op != DG_OP_SUMSQ) return DG_ERR_INVALID;
  if (rows < 0 || cols < 0) return DG_ERR_SHAPE;
  if (rows == 0 || cols == 0) return DG_OK;
  if (!X || !Y) return DG_ERR_INVALID;
  const bool out_bf16 = d->p.out_dtype == DG_BF16;
  if (!aligned(X, 4) || !aligned(Y, out_bf16 ? 2 : 4) || (w && !aligned(w, 2))) return DG_ERR_ALIGN;
  if (rows > (int64_t)0x7fffffff) return DG_ERR_SHAPE;
  hipStream_t st = (hipStream_t)stream;
  dg::RowsumArgs a = rowsum_args(d, X, nullptr, rows, cols);
  a.rms = 1;
  a.eps = eps;
  dg::NormArgs n;
  std::memset(&n, 0, sizeof n);
  n.X = X;
  n.rinv = nullptr;
  n.w = (const uint16_t*)w;
  n.Y = Y;
  n.rows = rows;
  n.cols = cols;
  n.out_bf16 = out_bf16;
  n.pre_round = d->p.norm_round == DG_NORM_PRE_WEIGHT;
  // one pass when the row fits in registers, else the reciprocal roots to a
  // workspace and a scaling pass
  if (dg::rmsnorm_fused_ok(a, n)) {
    if (dg::launch_rmsnorm_fused(a, n, st) != hipSuccess) return DG_ERR_HIP;
    return DG_OK;
  }
  void* ws = nullptr;
  dg_status s = get_workspace(st, (size_t)rows * sizeof(float), &ws);
  if (s != DG_OK) return s;
  a.out = (float*)ws;
  n.rinv = (const float*)ws;
  if (dg::launch_rowsum(a, st) != hipSuccess) return DG_ERR_HIP;
  if (dg::launch_rmsnorm_scale(n, st) != hipSuccess) return DG_ERR_HIP;
  return DG_OK;
}

dg_status dg_attn_desc_create(const dg_attn_params* p, dg_attn_desc** out) {
  if (!p || !out) return DG_ERR_INVALID;
  *out = nullptr;
  if (p->struct_size < sizeof(dg_attn_params)) return DG_ERR_INVALID;
  if (p->key_block < 1 || !in(p->causal, 0, 1) || (p->causal && p->q_block < 1)) return DG_ERR_INVALID;
  if (p->block_sum != DG_SEQ && p->block_sum != DG_TREE) return DG_ERR_INVALID;
  if (!in(p->p_dtype, DG_F32, DG_BF16) || !in(p->pv_fma, 0, 1) || !in(p->l_fma, 0, 1)) return DG_ERR_INVALID;
  if (!in(p->final_div, DG_ATTN_DIV, DG_ATTN_RECIP) || !in(p->out_dtype, DG_F32, DG_BF16)) return DG_ERR_INVALID;
  // the bf16 instruction takes the probabilities at bf16; the kernel's blocks
  // are whole 32-key instruction steps; a workgroup's 16-row waves share one split
  if (p->p_dtype != DG_BF16) return DG_ERR_UNSUPPORTED;
  if (p->key_block != 32 && p->key_block != 64 && p->key_block != 128) return DG_ERR_UNSUPPORTED;
  if (p->causal && p->q_block % 16 != 0) return DG_ERR_UNSUPPORTED;
  dg_attn_desc* d = new (std::nothrow) dg_attn_desc;
  if (!d) return DG_ERR_NOMEM;
  d->p = *p;
  d->p.struct_size = sizeof(dg_attn_params);
  if (!d->p.causal) d->p.q_block = 0;   // not part of an unmasked order
  *out = d;
  return DG_OK;
}

void dg_attn_desc_destroy(dg_attn_desc* d) { delete d; }

dg_status dg_attention(const dg_attn_desc* d, const void* Q, const void* K, const void* V, void* O, int64_t H,
                       int64_t Lq, int64_t Lk, int64_t dim, float qk_scale, void* stream) {
  if (!d) return DG_ERR_INVALID;
  if (H < 0 || Lq < 0 || Lk < 0 || dim < 0) return DG_ERR_SHAPE;
  if (!dg::attn_supported(dim, d->p.key_block)) return DG_ERR_UNSUPPORTED;
  if (H == 0 || Lq == 0) return DG_OK;
  if (Lk < 1 || H > 65535 || (d->p.causal && Lq != Lk)) return DG_ERR_SHAPE;
  if ((Lq + 15) / 16 > 65535) return DG_ERR_SHAPE;
  if (!Q || !K || !V || !O) return DG_ERR_INVALID;
  if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(O, 16)) return DG_ERR_ALIGN;
  dg::AttnArgs a;
  std::memset(&a, 0, sizeof a);
  a.Q = (const uint16_t*)Q;
  a.K = (const uint16_t*)K;
  a.V = (const uint16_t*)V;
  a.O = O;
  a.H = H;
  a.Lq = Lq;
  a.Lk = Lk;
  a.qk_scale = qk_scale;
  a.causal = d->p.causal;
  a.q_block = d->p.q_block;
  a.block_tree = d->p.block_sum == DG_TREE;
  a.pv_fma = d->p.pv_fma;
  a.l_fma = d->p.l_fma;
  a.final_recip = d->p.final_div == DG_ATTN_RECIP;
  a.out_bf16 = d->p.out_dtype == DG_BF16;
  if (dg::launch_attention(a, dim, d->p.key_block, (hipStream_t)stream) != hipSuccess) return DG_ERR_HIP;
  return DG_OK;
}

}  // extern "C"
