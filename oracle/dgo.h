/*
 * dgo.h -- CPU oracle for the descriptor-ordered GEMM and row reduction.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this code; only the tests, the smoke check and the benchmark's CPU
 * baseline do.  It shares no source with the GPU path.
 *
 * What it computes (paper: "Taming Bitwise Behavior in GPU Kernels with
 * Tensor Core", Sec. 3, the bit behaviour of parallel reductions):
 *
 *   A reduction is a dependence tree of binary32 additions; two kernels owe
 *   each other the same bits when their trees are equivalent up to swapping
 *   the children of a node (Sec. 3.1).  A matrix instruction folds
 *   instruction_k products and (optionally) the incoming accumulator into ONE
 *   rounding of their exact sum (Sec. 3.2.1).  A GEMM order is then fixed by
 *   the group width, whether the accumulator joins that rounding
 *   (use_fast_accum), where the short K turn falls (k_loop_step), the split-K
 *   cut points, how tiles and parts are combined and at which precision
 *   (partial_dtype / merge_dtype) (Sec. 3.2.2, the families of GEMM orders).
 *
 * The oracle evaluates exactly that order, one output at a time, with every
 * rounding explicit: exact group sums in a wide fixed-point accumulator,
 * binary32 round-to-nearest-even with gradual underflow, bfloat16 RNE.
 *
 * Storage: A is M x K bf16 row-major, B is K x N bf16 row-major, bias is N
 * bf16, C is M x N (fp32 or bf16 bits) row-major.  X is rows x cols fp32.
 */
#ifndef DGO_H
#define DGO_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { DGO_CARRY = 0, DGO_SEQ = 1, DGO_TREE = 2 };

/* Arithmetic of one matrix-instruction accumulator update.
 *  DGO_MODEL_EXACT  -- the paper's hypothesis (Sec. 3.2.1): the g products of
 *                      a group and (fma = 1) the accumulator are summed
 *                      exactly and rounded once.
 *  DGO_MODEL_GFX950 -- what the gfx950 bf16 MFMA instructions compute, as
 *                      read off the hardware with the paper's +L/-L/r
 *                      numerical experiments (Sec. 4): the group is folded
 *                      in chunks of 8 consecutive products; each chunk is
 *                      aligned to a fixed-point grid set by its largest
 *                      product, truncated, added to the accumulator and
 *                      rounded once (see dgo_chunk8). */
enum { DGO_MODEL_EXACT = 0, DGO_MODEL_GFX950 = 1 };
enum { DGO_EPI_NONE = 0, DGO_EPI_BIAS = 1, DGO_EPI_BIAS_SILU = 2 };

typedef struct {
  int32_t model;          /* DGO_MODEL_* */
  int32_t g;              /* products folded into one accumulator update (instruction_k) */
  int32_t tile_k;         /* accumulator-closing tile length inside a part (inner k_cut) */
  int32_t split_k;        /* number of parts S >= 1 (outer k_cut) */
  const int64_t* k_cuts;  /* S-1 strictly increasing interior cut points, or NULL for the span rule */
  int32_t tile_combine;   /* DGO_CARRY, DGO_SEQ or DGO_TREE */
  int32_t split_combine;  /* DGO_SEQ or DGO_TREE */
  int32_t tail_first;     /* 1: the short tile of a part comes first (k_loop_step) */
  int32_t fma;            /* 1: the accumulator joins the group's single rounding */
  int32_t partial_bf16;   /* 1: each part is rounded to bf16 before the merge */
  int32_t merge_bf16;     /* 1: every merge addition is rounded to bf16 */
  int32_t out_bf16;       /* 1: output stored as bf16 */
  int32_t epilogue;       /* DGO_EPI_* */
  int32_t pre_act_round;  /* 1: the pre-activation value is rounded to bf16 */
  int32_t leaf_w;         /* row reduction: elements per sequential leaf */
  int32_t sumsq;          /* row reduction: 1 = sum of squares */
  int32_t split_strided;  /* outer cut layout (Sec. 3.2.2, GEMV: layout): 0 contiguous
                             parts; 1 the axis is dealt in tiles of split_tile,
                             tile u going to part u mod S */
  int32_t split_tile;     /* width of a dealt tile (strided layout only) */
  int32_t leaf_strided;   /* row reduction leaf layout (Sec. 3.2.2, GEMV: layout):
                             0: leaf j holds elements [j leaf_w, (j+1) leaf_w);
                             1: leaf_w leaves (lanes), leaf j holding elements
                             j, j + leaf_w, j + 2 leaf_w, ... */
  int32_t fold_down;      /* how the leaves meet (Sec. 3.2.2 GEMV, Sec. 5.1):
                             0: balanced tree in leaf order (butterfly counting
                             its offsets up); 1: balanced tree over the leaves in
                             bit-reversed order (offsets counting down) */
  int32_t norm_pre_round; /* RMS normalisation: 1 = the normalised value is
                             rounded to bf16 before the weight multiplies it */
  int32_t in_f16;         /* GEMM operands A and B: 0 = bfloat16, 1 = IEEE binary16,
                             2 = OCP e4m3 codes (0..255 in each uint16; the gfx950
                             model then folds chunks of 16, dgo_chunk16_e4m3);
                             the bias stays bfloat16 */
} dgo_params;

/* Status: 0 ok, 1 invalid parameters, 3 shape inconsistent with the plan. */

/* Full GEMM.  C receives M*N fp32 values (out_bf16 = 0) or bf16 bits. */
int dgo_gemm(const dgo_params* p, const uint16_t* A, const uint16_t* B,
             const uint16_t* bias, void* C, int64_t M, int64_t N, int64_t K,
             int nthreads);

/* Column sums of a GEMM's output (the epilogue reduction the paper times,
 * Sec. 7): colsum[j] = the balanced tree (count-up, rows in order) over the
 * M output values of column j, each taken as stored (a bf16 output widened
 * exactly to fp32).  C holds M*N fp32 values or bf16 bits (out_bf16). */
int dgo_colsum(const void* C, int out_bf16, int64_t M, int64_t N, float* colsum, int nthreads);

/* Selected outputs (i[t], j[t]) of the same GEMM; out[t] is the output value
 * widened to fp32 (a bf16 output is exactly representable in fp32).  Row i of
 * A is read through A + i*K, so only the sampled rows need to exist. */
int dgo_gemm_at(const dgo_params* p, const uint16_t* A, const uint16_t* B,
                const uint16_t* bias, int64_t M, int64_t N, int64_t K,
                const int64_t* ii, const int64_t* jj, int64_t n, float* out,
                int nthreads);

/* Row reduction: out[r] for each of `rows` rows of X (row stride = cols). */
int dgo_rowsum(const dgo_params* p, const float* X, float* out, int64_t rows,
               int64_t cols, int nthreads);

/* RMS normalisation of each row, on the row's sum of squares s taken in the
 * descriptor's order (as dgo_rowsum with sumsq = 1):
 *   ms = RN32(s / n)  (n = cols as binary32),  v = RN32(ms + eps),
 *   q = RN32(sqrt(v)),  rinv = RN32(1 / q),  y_j = RN32(x_j * rinv),
 *   out_j = RN_out(RN32(y'_j * w_j)) with y'_j = y_j, or RN_bf16(y_j) when
 *   norm_pre_round;  without w (NULL), out_j = RN_out(y'_j).
 * w holds cols bf16 values; Y receives rows*cols fp32 values (out_bf16 = 0)
 * or bf16 bits.  rinv (if not NULL) receives each row's rinv. */
int dgo_rmsnorm(const dgo_params* p, const float* X, const uint16_t* w, float eps,
                void* Y, float* rinv, int64_t rows, int64_t cols, int nthreads);

/* Layer normalisation of each row, both row sums in the descriptor's leaf
 * order (leaf_w, leaf_strided, fold_down; the squares by the fma rule):
 *   s1 = sum of x_j,  mean = RN32(s1 / n),  d_j = RN32(x_j - mean),
 *   s2 = sum of squares of the d_j,  then as dgo_rmsnorm from s2:
 *   v = RN32(RN32(s2 / n) + eps), q = RN32(sqrt(v)), rinv = RN32(1 / q),
 *   y_j = RN32(d_j * rinv), y'_j = y_j or RN_bf16(y_j) (norm_pre_round),
 *   out_j = RN_out(RN32(RN32(y'_j * w_j) + b_j)), each of w, b optional
 *   (NULL: the step is left out).  w, b hold cols bf16 values. */
int dgo_layernorm(const dgo_params* p, const float* X, const uint16_t* w, const uint16_t* b,
                  float eps, void* Y, int64_t rows, int64_t cols, int nthreads);

/* Softmax of each row:  m = the row's largest element (a NaN anywhere makes
 * it NaN; exact, so independent of order),  e_j = dgo_exp(RN32(x_j - m)),
 * s = the sum of the e_j in the descriptor's leaf order (as dgo_rowsum with
 * sumsq = 0),  rinv = RN32(1 / s),  out_j = RN_out(RN32(e_j * rinv)).
 * Y receives rows*cols fp32 values (out_bf16 = 0) or bf16 bits. */
int dgo_softmax(const dgo_params* p, const float* X, void* Y, int64_t rows, int64_t cols,
                int nthreads);

/* The count-down butterfly's tree over lanes 0..P-1 (P rounded up to a power
 * of two), lane j < n holding v[j], lanes from n on empty.  Exposed for tests. */
float dgo_tree_bitrev(const float* v, int n, int P);

/* One accumulator update over n products a[t]*b[t] (n <= g; the rest of the
 * group is zero padding) under the given model and fma rule.  Exposed for
 * tests. */
float dgo_group_update(int model, float acc, const uint16_t* a, const uint16_t* b,
                       int n, int g, int fma);

/* Batch of independent updates: out[t] = dgo_group_update(model, acc[t],
 * a + t*n, b + t*n, n, g, fma) for t < count, with binary16 operands when
 * f16 = 1. */
void dgo_group_update_batch(int model, int64_t count, const float* acc,
                            const uint16_t* a, const uint16_t* b, int n, int g,
                            int fma, float* out, int nthreads, int f16);

/* One gfx950 MFMA chunk update: acc and n <= 8 products of bf16 operands
 * (dgo_chunk8) or of either operand format (f16 = 1: binary16). */
float dgo_chunk8(float acc, const uint16_t* a, const uint16_t* b, int n);
float dgo_chunk8_fmt(int f16, float acc, const uint16_t* a, const uint16_t* b, int n);
/* One 16-product chunk of a gfx950 fp8 MFMA (e4m3 codes as uint16 0..255;
 * n <= 16 real products, the rest zero padding). */
float dgo_chunk16_e4m3(float acc, const uint16_t* a, const uint16_t* b, int n);

/* Exact sum of n products plus c, rounded once to binary32 (RNE). */
float dgo_exact_dot_rn32(float c, const uint16_t* a, const uint16_t* b, int n);
float dgo_exact_dot_rn32_fmt(int f16, float c, const uint16_t* a, const uint16_t* b, int n);

/* Balanced tree over n binary32 values (level-wise pairing, odd last carried). */
float dgo_tree(const float* v, int n, int bf16_round);

/* Rounding helpers. */
uint16_t dgo_f32_to_bf16(float x);
float dgo_bf16_to_f32(uint16_t h);
float dgo_f16_to_f32(uint16_t h);   /* exact */

/* Epilogue functions: the exp and SiLU the descriptor's epilogue uses. */
float dgo_exp(float x);
float dgo_silu(float z);
/* e[i] = dgo_exp(x), s[i] = dgo_silu(x) for the binary32 x with bits start + i. */
void dgo_exp_silu_range(uint64_t start, int64_t count, float* e, float* s, int nthreads);

/* ---------------------------------------------------------------- attention
 *
 * The reduction order of one attention head (App. F): per query row i, the
 * keys are walked in blocks; the kernel carries a running maximum m, a
 * denominator l and an output row O (binary32).  At block j (keys kb..ke-1):
 *   s_t   = RN32(score_t * qk_scale), score_t = q_i . k_t by the first matrix
 *           multiplication (groups of 32 over the head dimension from +0,
 *           accumulator carried); a masked key adds ATTN_MASK_OFFSET (-1e6);
 *   mn    = max(m, max_t s_t)            (exact);
 *   alpha = exp2(RN32(m - mn)),  p_t = exp2(RN32(s_t - mn))  (dgo_exp2);
 *   rs    = the block's p_t summed by block_sum: chain in key order, or the
 *           balanced tree over the block's positions in key order;
 *   l     = fma(alpha, l, rs)  (l_fma)  or  RN32(RN32(alpha l) + rs);
 *   O_c   = the block's P.V over its keys in groups of 32 from the block
 *           start, p narrowed to bf16, with RN32(alpha O_c) as the
 *           accumulator (pv_fma) or from +0 and then added to RN32(alpha O_c);
 *   m     = mn;
 * starting from m = -inf, l = +0, O = +0; finally out_c = RN_out(O_c / l)
 * or, with final_recip, RN_out(O_c * RN32(1 / l)).  The blocks: see
 * attn_blocks in dgo.c (unmasked: width key_block from key 0; causal: the
 * split at the multiples of q_block). */
typedef struct {
  int32_t key_block;     /* w, keys per block (BLOCK_N) */
  int32_t causal;        /* 1: key t visible to query i iff t <= i (Lq = Lk) */
  int32_t q_block;       /* BLOCK_M: where the masked stage starts (causal only) */
  int32_t block_sum;     /* DGO_SEQ or DGO_TREE */
  int32_t pv_fma;        /* 1: rescaled output row is the P.V accumulator */
  int32_t l_fma;         /* 1: the denominator update is one fused multiply-add */
  int32_t final_recip;   /* 0: out = O / l;  1: out = O * (1 / l) */
  int32_t out_bf16;      /* output stored as bf16 */
  int32_t model;         /* DGO_MODEL_* for both matrix multiplications */
} dgo_attn_params;

/* Q: H x Lq x d, K and V: H x Lk x d, bf16 row-major; O: H x Lq x d (fp32
 * values or bf16 bits).  Status 1: invalid parameters; 3: shapes (Lk = 0,
 * d = 0, or a causal mask with Lq != Lk). */
int dgo_attention(const dgo_attn_params* p, const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                  void* O, int64_t H, int64_t Lq, int64_t Lk, int64_t d, float qk_scale, int nthreads);
/* Selected rows (hh[r], ii[r]): out[r * d + c] as binary32 (bf16 outputs widened). */
int dgo_attention_rows(const dgo_attn_params* p, const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                       int64_t H, int64_t Lq, int64_t Lk, int64_t d, float qk_scale, const int64_t* hh,
                       const int64_t* ii, int64_t n, float* out, int nthreads);
/* 2^x by the library's fixed steps (see dgo.c), and over a range of bit patterns. */
float dgo_exp2(float x);
void dgo_exp2_range(uint64_t start, int64_t count, float* out, int nthreads);

/* Cut plan for (K, params): writes S+1 cut points to cuts (caller provides
 * split_k + 1 slots).  Returns 0 or a status. */
int dgo_plan_cuts(const dgo_params* p, int64_t K, int64_t* cuts);

#ifdef __cplusplus
}
#endif
#endif
