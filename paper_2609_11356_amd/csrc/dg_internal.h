// dg_internal.h -- library-internal types shared by the host API and kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/dg.h"

struct dg_desc {
  dg_desc_params p;            // validated copy; p.k_cuts points into cuts[]
  int64_t cuts[DG_MAX_SPLIT];  // explicit interior cuts (n_cuts of them)
  int group;                   // products per instruction group (32 or 16)
  char sig[2048];              // canonical order text (every cut written out)
};

struct dg_attn_desc {
  dg_attn_params p;            // validated copy
};

namespace dg {

// Everything a GEMM launch needs, passed by value as the kernel argument.
struct GemmArgs {
  const uint16_t* A;
  const uint16_t* B;
  const uint16_t* bias;
  void* C;
  float* ws;                     // split-K partials [S][M][N] (fp32 storage)
  int64_t M, N, K;
  int64_t cuts[DG_MAX_SPLIT + 1];
  int32_t S;
  int32_t tile_k, group, tile_combine, tail_first, fma;
  int32_t partial_bf16, out_bf16, epilogue, pre_act;
  int32_t order;                 // block order of the v3 kernels (speed only)
  int64_t split_w;               // strided split: dealt tile width (0: contiguous parts)
  int64_t n_split;               // mixed-width ping-pong: first column of the 192-wide blocks
  int32_t in_f16;                // operands A and B are binary16 (else bfloat16)
  int32_t b_e4m3;                // B holds one OCP e4m3 byte per element (A bf16)
  int32_t ab_e4m3;               // A and B hold OCP e4m3 bytes (the fp8 instructions)
  float* colsum_part;            // set (single part, 256-row blocks): column sums of each 256-row
                                 // run of C, [ceil(M / 256)][N], folded in the epilogue
};

struct CombineArgs {
  const float* ws;
  const uint16_t* bias;
  void* C;
  int64_t M, N;
  int32_t S;
  int32_t split_combine, merge_bf16, out_bf16, epilogue, pre_act;
};

struct RowsumArgs {
  const float* X;
  float* out;
  int64_t rows, cols;
  int32_t leaf_w, sumsq, fma;
  int32_t strided, down;         // leaf layout and lane fold
  int32_t rms;                   // 1: out[row] = the RMS-norm reciprocal root of the sum,
                                 // 2: out[row] = 1 / sum, 3: out[row] = sum / cols
  float eps;
};

struct NormArgs {
  const float* X;
  const float* rinv;             // per row
  const uint16_t* w;             // bf16 weight or null
  const uint16_t* b;             // bf16 bias or null
  void* Y;
  int64_t rows, cols;
  int32_t out_bf16, pre_round;
};

struct ColsumArgs {
  const void* C;                 // M x N output, fp32 or bf16
  float* part;                   // [nchunk][N] subtree roots (nchunk > 1)
  float* colsum;                 // N
  int64_t M, N;
  int32_t out_bf16;
};

struct AttnArgs {
  const uint16_t* Q;             // H x Lq x d bf16
  const uint16_t* K;             // H x Lk x d bf16
  const uint16_t* V;             // H x Lk x d bf16
  void* O;                       // H x Lq x d, fp32 or bf16
  int64_t H, Lq, Lk;
  float qk_scale;
  int32_t causal, q_block;
  int32_t block_tree, pv_fma, l_fma, final_recip, out_bf16;
};

bool attn_supported(int64_t d, int key_block);
hipError_t launch_attention(const AttnArgs& a, int64_t d, int key_block, hipStream_t s);

// This device's copy of the fixed split-K scratch array of dg_gemm_noalloc
// (DG_NOALLOC_SCRATCH_BYTES), looked up once per device with that device
// current; never allocates.
hipError_t noalloc_scratch(void** out);

// launchers (return hipSuccess or the launch error)
hipError_t launch_gemm_generic(const GemmArgs& a, hipStream_t s);
hipError_t launch_gemm_scalar(const GemmArgs& a, hipStream_t s);   // groups of one (scalar FMA)
hipError_t launch_gemm_tiled(const GemmArgs& a, int tile_m, int tile_n, hipStream_t s);
bool tiled_supported(int tile_m, int tile_n);
hipError_t launch_gemm_v3(const GemmArgs& a, int tile_m, int tile_n, int occupancy, hipStream_t s);
bool v3_supported(int tile_m, int tile_n, int occupancy);
// tile chain or tree, or fma = 0, on 128 x 64 tiled blocks (levels: the
// tree's stack depth, 2..7; each part at most 2^levels tiles)
hipError_t launch_gemm_tc(const GemmArgs& a, int levels, hipStream_t s);
// e4m3 x e4m3 with a carried accumulator and fma = 1 on the block-scaled fp8
// instructions (K, N and the part starts multiples of 16; A, B, C 16-byte
// aligned): tile 128, 128 x 128 blocks on 128-k slabs; tile 256, 256 x 256
// blocks on 64-k slabs loaded direct to LDS (M K and K N below 2^31 bytes)
hipError_t launch_gemm_f8(const GemmArgs& a, int tile, hipStream_t s);
// bf16 on the same four-wave ring: 256 x 128 blocks, two per CU, 32-k slabs
// loaded direct to LDS (the tiled layout's conditions; M K and K N below
// 2^30 elements)
hipError_t launch_gemm_b16n(const GemmArgs& a, hipStream_t s);
hipError_t launch_gemm_wide(const GemmArgs& a, int tile_m, int tile_n, hipStream_t s);
bool wide_supported(int tile_m, int tile_n);
bool wide_is_pp(int tile_m, int tile_n);   // the ping-pong kernel (buffer-resource offsets)
hipError_t launch_gemm_pp_mixed(const GemmArgs& a, hipStream_t s);   // n_split set
// direct-to-LDS ping-pong: 256 x 256 blocks, or (mixed) the kernel-6 split
hipError_t launch_gemm_ppd(const GemmArgs& a, bool mixed, hipStream_t s);
hipError_t launch_gemm_w4(const GemmArgs& a, hipStream_t st);
hipError_t launch_gemm_skinny(const GemmArgs& a, int tile_m, int tile_n, int depth, int slab_k, hipStream_t s);
bool skinny_supported(int tile_m, int tile_n, int depth, int slab_k);
hipError_t launch_gemm_skinny_dma(const GemmArgs& a, int tile_m, int tile_n, int slots, int slab_k, hipStream_t s);
// packed B (dg_panel.hip): the layout writer, and the few-row kernel on it
// (tms 16-row A tiles per wave, a ring of depth k blocks; avec: A rows read
// as 16-byte runs, else element by element)
hipError_t launch_pack_b(const uint16_t* B, uint16_t* Bp, int64_t K, int64_t N, hipStream_t s);
hipError_t launch_pack_b8(const uint8_t* B, uint8_t* Bp, int64_t K, int64_t N, hipStream_t s);
hipError_t launch_gemm_panel(const GemmArgs& a, int tms, int depth, bool avec, hipStream_t s);
bool panel_supported(int tms, int depth, bool avec, bool b8);
int panel_default_depth(int tms, bool avec, bool b8);
bool skinny_dma_supported(int tile_m, int tile_n, int slots, int slab_k);
hipError_t launch_splitk_combine(const CombineArgs& a, hipStream_t s);
hipError_t launch_rowsum(const RowsumArgs& a, hipStream_t s);
hipError_t launch_rmsnorm_scale(const NormArgs& a, hipStream_t s);
bool rmsnorm_fused_ok(const RowsumArgs& r, const NormArgs& a);
hipError_t launch_rmsnorm_fused(const RowsumArgs& r, const NormArgs& a, hipStream_t s);
// softmax: one pass (strided lanes, row in registers), or the shifted
// exponentials of each row into a.Y (fp32) for the three-pass path
bool softmax_fused_ok(const RowsumArgs& r, const NormArgs& a);
hipError_t launch_softmax_fused(const RowsumArgs& r, const NormArgs& a, hipStream_t s);
hipError_t launch_softmax_exp(const NormArgs& a, hipStream_t s);
// layer normalisation: one pass (strided lanes, row in registers), or the
// centred values into a.Y given the means in a.rinv (three-pass path)
hipError_t launch_layernorm_fused(const RowsumArgs& r, const NormArgs& a, hipStream_t s);
hipError_t launch_layernorm_center(const NormArgs& a, hipStream_t s);
// column sums of a GEMM output: subtrees of 256 rows, then their tree
hipError_t launch_colsum(const ColsumArgs& a, hipStream_t s);
hipError_t launch_colsum_merge(const ColsumArgs& a, hipStream_t s);   // run roots in a.part only

}  // namespace dg
