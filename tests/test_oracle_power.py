"""Power of the oracle's pins: plausible mistakes planted in a copy of the
oracle's C source must each be caught by at least one pin (the paper checks
its own byte comparisons against a deliberately broken kernel, App. E).
CPU only; the planted copies live in a temporary directory."""
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle
from tests import test_oracle_attention as attn
from tests import test_oracle_fp8 as fp8
from tests import test_oracle_pins as pins

HERE = os.path.dirname(os.path.abspath(oracle.__file__))

MUTANTS = {
    "drops the last group of a tile": (
        "for (int64_t q = t0; q < t0 + tl; q += p->g) {",
        "for (int64_t q = t0; q + p->g < t0 + tl; q += p->g) {"),
    "merges the parts last to first": (
        "  float s = v[0];\n  for (int k = 1; k < n; ++k) { s = s + v[k]; if (bf16_round) s = rnbf(s); }",
        "  float s = v[n - 1];\n  for (int k = n - 2; k >= 0; --k) { s = s + v[k]; if (bf16_round) s = rnbf(s); }"),
    "tree counts down (pairs k with k + n/2)": (
        "float s = t[2 * k] + t[2 * k + 1];",
        "float s = t[k] + t[k + h];"),
    "products truncate toward -inf": (
        "else m = (qe - e) >= 64 ? 0 : m >> (qe - e);",
        "else m = (qe - e) >= 64 ? (neg ? 1 : 0) : (neg ? (m + ((uint64_t)1 << (qe - e)) - 1) >> (qe - e) : m >> (qe - e));"),
    "product window one bit wider": ("#define CHUNK_W 24", "#define CHUNK_W 25"),
    "result grid one bit coarser": ("#define CHUNK_F 31", "#define CHUNK_F 30"),
    "accumulator left out of the chunk sum": (
        "    split_f32(acc, &neg, &m, &e);\n    xacc_add_int(&x, neg, m, e);\n  }\n  /* leading bit",
        "    split_f32(acc, &neg, &m, &e);\n    (void)m;\n  }\n  /* leading bit"),
    "fma flag ignored": ("  s = fma ? acc : 0.0f;", "  s = acc; fma = 1;"),
    "short tile always last": ("if (p->tail_first && len % tk)", "if (0 && len % tk)"),
    "pre-activation rounding skipped": ("if (p->pre_act_round) z = rnbf(z);", "if (0) z = rnbf(z);"),
    "B read transposed": ("bbuf[u] = bcol[idx[q + u] * c->ldb];", "bbuf[u] = bcol[idx[q + u]];"),
    "strided tiles dealt to the next part": ("for (int64_t u = s; u * w < K; u += S)",
                                             "for (int64_t u = (s + 1) % S; u * w < K; u += S)"),
    "strided tile width halved": ("const int64_t w = p->split_tile;", "const int64_t w = p->split_tile / 2;"),
    "bf16 conversion truncates": (
        "return (uint16_t)((u + 0x7fffu + lsb) >> 16);", "(void)lsb; return (uint16_t)(u >> 16);"),
    "strided leaves take consecutive elements": ("int64_t step = strided ? W : 1;", "int64_t step = 1;"),
    "count-down fold taken in leaf order": ("if (p->fold_down) return dgo_tree_bitrev(leaves, (int)L, (int)lanes);",
                                            "if (p->fold_down) return dgo_tree(leaves, (int)L, 0);"),
    "bit reversal one bit short": ("while ((1 << b) < P) ++b;", "while ((2 << b) < P) ++b;"),
    "empty lane adds zero": ("t[k] = (hl && hr) ? l + r : (hl ? l : r);", "t[k] = l + r;"),
    "mean over cols - 1": ("const float n = (float)cols;\n  if (nthreads < 1)",
                           "const float n = (float)(cols - 1);\n  if (nthreads < 1)"),
    "eps added after the root": ("float v = ms + eps;\n      float q = sqrtf(v);",
                                 "float v = ms;\n      float q = sqrtf(v) + eps;"),
    "weight before the bf16 rounding": (
        "if (p->norm_pre_round) y = rnbf(y);\n        if (w) y = y * dgo_bf16_to_f32(w[j]);\n        if (p->out_bf16)",
        "if (w) y = y * dgo_bf16_to_f32(w[j]);\n        if (p->norm_pre_round) y = rnbf(y);\n        if (p->out_bf16)"),
    "rmsnorm sums the row in index order": ("float s = row_reduce(p, x, cols, leaves);",
                                            "float s = 0.0f;\n      for (int64_t k = 0; k < cols; ++k) s = fmaf(x[k], x[k], s);"),
    "softmax without the max shift": ("for (int64_t j = 0; j < cols; ++j) e[j] = dgo_exp(x[j] - m);",
                                      "for (int64_t j = 0; j < cols; ++j) e[j] = dgo_exp(x[j]);"),
    "softmax divides instead of multiplying": ("float y = e[j] * rinv;", "float y = e[j] / s;"),
    "softmax sums in index order": ("float s = row_reduce(p, e, cols, leaves);",
                                    "float s = 0.0f;\n      for (int64_t j = 0; j < cols; ++j) s = s + e[j];"),
    "layernorm squares the uncentred values": ("for (int64_t j = 0; j < cols; ++j) d[j] = x[j] - mean;",
                                               "for (int64_t j = 0; j < cols; ++j) d[j] = x[j] - 0.0f * mean;"),
    "layernorm bias before the weight": (
        "if (w) y = y * dgo_bf16_to_f32(w[j]);\n        if (b) y = y + dgo_bf16_to_f32(b[j]);",
        "if (b) y = y + dgo_bf16_to_f32(b[j]);\n        if (w) y = y * dgo_bf16_to_f32(w[j]);"),
    "layernorm variance over cols - 1": ("float var = s2 / n;", "float var = s2 / (n - 1.0f);"),
    "SUMSQ fma never fused": ("else if (p->fma) s = fmaf(x[k], x[k], s);", "else if (0) s = fmaf(x[k], x[k], s);"),
    "exp polynomial one term short": ("  p = fmaf(p, r, (float)(1.0 / 720.0));\n", ""),
    "sign of a product lost": ("int sign = (a[t] >> 15) ^ (b[t] >> 15);\n    if (op_isnan(a[t], f16)",
                               "int sign = 0;\n    if (op_isnan(a[t], f16)"),
    "part stored without its bf16 rounding": ("pvals[s] = p->partial_bf16 ? rnbf(v) : v;", "pvals[s] = v;"),
    "chained merge without its bf16 rounding": (
        "for (int k = 1; k < n; ++k) { s = s + v[k]; if (bf16_round) s = rnbf(s); }",
        "for (int k = 1; k < n; ++k) { s = s + v[k]; }"),
    "tree merge without its bf16 rounding": ("t[k] = bf16_round ? rnbf(s) : s;", "t[k] = s;"),
    "merge rounded to bf16 only at the end": (
        "for (int k = 1; k < n; ++k) { s = s + v[k]; if (bf16_round) s = rnbf(s); }",
        "for (int k = 1; k < n; ++k) { s = s + v[k]; }\n  if (bf16_round) s = rnbf(s);"),
    "attention rescale skipped": ("const float alpha = dgo_exp2(m - mn);",
                                  "const float alpha = m == -INFINITY ? 0.0f : 1.0f;"),
    "attention key block one wider": ("const int64_t w = p->key_block;\n  int64_t n = 0;",
                                      "const int64_t w = p->key_block + 1;\n  int64_t n = 0;"),
    "attention probabilities truncated to bf16": ("pb[u] = dgo_f32_to_bf16(pr[u]);",
                                                  "pb[u] = (uint16_t)(f2u(pr[u]) >> 16);"),
    "attention denominator fma ignored": ("l = p->l_fma ? fmaf(alpha, l, rs) : alpha * l + rs;",
                                          "l = alpha * l + rs;"),
    "attention final reciprocal ignored": ("if (p->final_recip) {\n    const float r = 1.0f / l;",
                                           "if (0) {\n    const float r = 1.0f / l;"),
    "attention causal split on the key grid": ("const int64_t q0 = i / p->q_block * p->q_block;",
                                               "const int64_t q0 = i / p->key_block * p->key_block;"),
    "attention mask offset left out": ("if (st2[b] && t > i) v = v + ATTN_MASK_OFFSET;", "if (0) v = v;"),
    "attention block sum always a chain": (
        "const float rs = p->block_sum == DGO_TREE ? dgo_tree(pr, (int)n, 0) : chain(pr, (int)n, 0);",
        "const float rs = chain(pr, (int)n, 0);"),
    "attention P.V restarts from zero": ("float acc = p->pv_fma ? base : 0.0f;", "float acc = 0.0f;"),
    "attention score scaled before the dot product ends": ("float v = acc * qk_scale;",
                                                           "float v = acc * qk_scale * 1.0000001f;"),
    "exp2 polynomial one term short": ("  p = fmaf(p, f, c6);\n", ""),
    "binary16 exponent bias off by one": ("bias = f16 == 2 ? 7 : f16 ? 15 : 127;",
                                          "bias = f16 == 2 ? 7 : f16 ? 14 : 127;"),
    "e4m3 exponent bias off by one": ("bias = f16 == 2 ? 7 : f16 ? 15 : 127;",
                                      "bias = f16 == 2 ? 8 : f16 ? 15 : 127;"),
    "fp8 group grid one bit coarser": ("#define F8_GW 13", "#define F8_GW 12"),
    "fp8 chunk grid one bit finer": ("#define F8_W 24", "#define F8_W 25"),
    "fp8 result grid one bit finer": ("#define F8_F 31", "#define F8_F 32"),
    "fp8 accumulator kept one binade lower": ("#define F8_DROP 25", "#define F8_DROP 26"),
    "fp8 accumulator never left out": ("    if (xacc_lead >= E - F8_DROP) xacc_add_int(&x, neg, m, e);",
                                       "    (void)xacc_lead; xacc_add_int(&x, neg, m, e);"),
    "fp8 chunks of 8 products": ("const int cw = (f16 == 2) ? 16 : 8;", "const int cw = 8;"),
    "fp8 group sums truncated toward zero": (
        "return v >= 0 ? (v >> s) : -((-v + ((int64_t)1 << s) - 1) >> s);",
        "return v >= 0 ? (v >> s) : -((-v) >> s);"),
    "binary16 product scale off by one": ("const int fb2 = 2 * op_frac(f16);",
                                          "const int fb2 = 2 * op_frac(f16) - f16;"),
}

CHECKS = [
    lambda: pins.test_bf16_rounding_matches_torch(),
    lambda: pins.test_exact_dot_matches_rationals("spread"),
    lambda: pins.test_group_of_one_is_sequential_fp32_dot(1),
    lambda: [pins.test_all_ones_counts_terms(d, K) for d in pins.DESCS[:5] for K in (257, 576)],
    lambda: pins.test_splitk_walk_gfx950_matches_paper(),
    lambda: pins.test_nonassociativity_hand_examples(),
    lambda: pins.test_tree_is_recursive_halving_over_negzero_padding(),
    lambda: pins.test_rowsum_special_cases(),
    lambda: pins.test_tiles_of_one_group_seq_equals_carry_without_fma("gfx950", 32),
    lambda: pins.test_fma_on_ignores_instruction_shape_on_gfx950(),
    lambda: pins.test_explicit_cuts_equal_span_rule_and_tail_position(),
    lambda: pins.test_exp_accuracy_dense_sweep(),
    lambda: pins.test_epilogue_rounding_points(),
    lambda: pins.test_chunk_model_hand_examples(),
    lambda: pins.test_strided_layout_hand_walk("gfx950"),
    lambda: pins.test_strided_small_integers_are_exact(4, 64, 32, 4096),
    lambda: pins.test_fold_down_hand_example(),
    lambda: pins.test_folds_match_simulated_butterflies(),
    lambda: pins.test_strided_leaves_take_every_count_th_element(),
    lambda: pins.test_strided_special_cases(),
    lambda: pins.test_rmsnorm_hand_example(),
    lambda: pins.test_rmsnorm_closed_forms(),
    lambda: pins.test_rmsnorm_follows_the_rowsum_order_and_rounding_points(),
    lambda: pins.test_softmax_closed_forms(),
    lambda: pins.test_softmax_steps_and_rounding_points(),
    lambda: pins.test_layernorm_closed_forms(),
    lambda: pins.test_layernorm_steps_and_rounding_points(),
    lambda: pins.test_bf16_parts_and_merges_hand_examples(),
    lambda: pins.test_bf16_parts_and_merges_match_rationals(4, "tree", "bf16", "bf16"),
    lambda: pins.test_f16_decoding_matches_numpy_on_every_pattern(),
    lambda: attn.test_exp2_exact_points_and_edges(),
    lambda: attn.test_exp2_accuracy_dense_sweep(),
    lambda: [attn.test_recurrence_matches_rationals(di) for di in (0, 21, 45, 66, 93, 120)],
    lambda: [attn.test_equal_scores_give_the_mean_of_the_visible_values(di) for di in (0, 44, 92)],
    lambda: [attn.test_one_dominant_key_returns_its_value_row(di) for di in (1, 53, 93)],
    lambda: attn.test_query_block_enters_only_causal_answers_off_the_key_grid(),
    lambda: pins.test_f16_exact_dot_is_the_rational_sum_rounded_once(),
    lambda: pins.test_f16_chunk_model_hand_examples(),
    lambda: pins.test_f16_chunk_model_equals_exact_when_window_holds_everything(),
    lambda: [fp8.test_hand_examples(c) for c in range(len(fp8.HAND))],
    lambda: [fp8.test_walk_matches_the_placement_rule(r) for r in fp8.WALK_R],
    lambda: fp8.test_equals_exact_when_the_grids_hold_everything("16x16x32_fp8"),
    lambda: fp8.test_fma_on_ignores_the_instruction_shape(),
]


def _build_mutant(tmp, old, new):
    src = open(os.path.join(HERE, "dgo.c")).read()
    assert src.count(old) == 1, "mutation site not found exactly once: %r" % old[:60]
    d = tmp / "m"
    d.mkdir()
    shutil.copy(os.path.join(HERE, "dgo.h"), d / "dgo.h")
    (d / "dgo.c").write_text(src.replace(old, new))
    lib = d / "libdgo.so"
    subprocess.run(["gcc", "-std=gnu11", "-O2", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
                    "-o", str(lib), str(d / "dgo.c"), "-lm"], check=True, capture_output=True)
    return str(lib)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(name, tmp_path):
    lib = _build_mutant(tmp_path, *MUTANTS[name])
    prev = oracle.use_library(lib)
    caught = []
    try:
        for i, check in enumerate(CHECKS):
            try:
                check()
            except (AssertionError, oracle.OracleError):
                caught.append(i)
                break
    finally:
        oracle.restore_library(prev)
    assert caught, "no pin caught the planted mistake: " + name


def test_unmutated_oracle_passes_every_check():
    for check in CHECKS:
        check()
