"""Planted mistakes in the oracle must be caught by its pins.

Each mutant is a one-line textual change to ``oracle/lsa_oracle.c`` -- a
reversed tie-break, a dropped scale, a wrong sign, a wrong token or dimension
index, a dropped term -- compiled on the CPU into a throw-away library.  The
test passes when at least one pin fails for every mutant, which shows the pins
can tell a plausible slip in the oracle from the real thing.
"""
import os
import subprocess
import tempfile

import pytest

import oracle
import oracle_pins as P

SRC = os.path.join(os.path.dirname(oracle.__file__), "lsa_oracle.c")

MUTANTS = {
    "top_p_strict_mass": ("if ((unsigned __int128)cum * (uint64_t)p_den >= need) break;",
                          "if ((unsigned __int128)cum * (uint64_t)p_den > need) break;"),
    "top_p_tie_reversed": ("  return (x->c > y->c) - (x->c < y->c);\n}\n\n/*\n * Top-p set",
                           "  return (x->c < y->c) - (x->c > y->c);\n}\n\n/*\n * Top-p set"),
    "top_p_least_probable_first": ("  if (x->s > y->s) return -1;\n  if (x->s < y->s) return 1;\n"
                                   "  return (x->c > y->c) - (x->c < y->c);\n}\n\n/*\n * Top-p set",
                                   "  if (x->s > y->s) return 1;\n  if (x->s < y->s) return -1;\n"
                                   "  return (x->c > y->c) - (x->c < y->c);\n}\n\n/*\n * Top-p set"),
    "top_p_mass_not_summed": ("    Z += q[s];\n", "    Z = q[s];\n"),
    "exp_fixed_no_low_part": ("  r = fmaf(-k, ln2_lo, r);\n", ""),
    "exp_fixed_short_series": ("for (int j = 1; j < 8; ++j) p = fmaf(p, r, inv_fact[j]);",
                               "for (int j = 1; j < 7; ++j) p = fmaf(p, r, inv_fact[j]);"),
    "golden_vote_strict": ("if (votes[s] >= theta) {", "if (votes[s] > theta) {"),
    "golden_union_last_step": ("    memset(votes, 0, (size_t)n * sizeof *votes);\n",
                               "    memset(votes, 0, (size_t)n * sizeof *votes);\n    memset(label, 0, (size_t)n);\n"),
    "tie_break_reversed_f": ("  return (x->c > y->c) - (x->c < y->c);\n}\n\nstatic int by_score_desc_i",
                             "  return (x->c < y->c) - (x->c > y->c);\n}\n\nstatic int by_score_desc_i"),
    "tie_break_reversed_i": ("  return (x->c > y->c) - (x->c < y->c);\n}\n\nstatic int ascending_i32",
                             "  return (x->c < y->c) - (x->c > y->c);\n}\n\nstatic int ascending_i32"),
    "smallest_first": ("  if (x->s > y->s) return -1;\n  if (x->s < y->s) return 1;\n  return (x->c > y->c) - (x->c < y->c);\n}\n\nstatic int by_score_desc_i",
                       "  if (x->s > y->s) return 1;\n  if (x->s < y->s) return -1;\n  return (x->c > y->c) - (x->c < y->c);\n}\n\nstatic int by_score_desc_i"),
    "output_not_ascending": ("  free(v);\n  qsort(out, (size_t)k, sizeof *out, ascending_i32);\n  return k;\n}\n\n/* Top-k of int64",
                             "  free(v);\n  return k;\n}\n\n/* Top-k of int64"),
    "score_f32_dropped_term": ("for (int32_t i = 0; i < D; ++i) s += (double)qe[i]",
                               "for (int32_t i = 1; i < D; ++i) s += (double)qe[i]"),
    "score_bf16_wrong_sign": ("s += bf16_to_f64(qe[i]) * bf16_to_f64(E[c * D + i]);",
                              "s -= bf16_to_f64(qe[i]) * bf16_to_f64(E[c * D + i]);"),
    "score_i8_reversed_dims": ("(int64_t)qe[i] * (int64_t)E[c * D + i]",
                               "(int64_t)qe[i] * (int64_t)E[c * D + (D - 1 - i)]"),
    "union_drops_last_list": ("j < (int64_t)n_lists * k; ++j", "j < (int64_t)(n_lists - 1) * k; ++j"),
    "attn_dropped_scale": ("logit[i] = dot * scale;", "logit[i] = dot;"),
    "attn_exp_wrong_sign": ("logit[i] = exp(logit[i] - m);", "logit[i] = exp(m - logit[i]);"),
    "attn_k_token_index": ("const int64_t tok = (int64_t)sel[i / C] * C + i % C;\n      double dot",
                           "const int64_t tok = (int64_t)sel[i / C] + i % C;\n      double dot"),
    "attn_v_token_index": ("const int64_t tok = (int64_t)sel[i / C] * C + i % C;\n        acc",
                           "const int64_t tok = (int64_t)sel[i / C] + i % C;\n        acc"),
    "attn_k_transposed_dims": ("bf16_to_f64(Kh[tok * d + e])", "bf16_to_f64(Kh[tok * d + (d - 1 - e)])"),
    "attn_v_transposed_dims": ("bf16_to_f64(Vh[tok * d + e])", "bf16_to_f64(Vh[tok * d + (d - 1 - e)])"),
    "attn_lse_dropped_max": ("    lse[r] = m + log(Z);\n  }\n  free(logit);", "    lse[r] = log(Z);\n  }\n  free(logit);"),
    "attn_unnormalised": ("      out[(int64_t)r * d + e] = acc / Z;\n    }\n    lse[r] = m + log(Z);\n  }\n  free(logit);",
                          "      out[(int64_t)r * d + e] = acc;\n    }\n    lse[r] = m + log(Z);\n  }\n  free(logit);"),
    "tokens_lse_dropped_max": ("    lse[r] = m + log(Z);\n  }\n  free(w);", "    lse[r] = log(Z);\n  }\n  free(w);"),
    "tokens_unnormalised": ("      out[(int64_t)r * d + e] = acc / Z;\n    }\n    lse[r] = m + log(Z);\n  }\n  free(w);",
                            "      out[(int64_t)r * d + e] = acc;\n    }\n    lse[r] = m + log(Z);\n  }\n  free(w);"),
    "attn_empty_lse_zero": ("  if (nsel == 0) { /* nothing to attend: the empty sum */\n"
                            "    for (int64_t i = 0; i < (int64_t)R * d; ++i) out[i] = 0.0;\n"
                            "    for (int32_t r = 0; r < R; ++r) lse[r] = -INFINITY;",
                            "  if (nsel == 0) { /* nothing to attend: the empty sum */\n"
                            "    for (int64_t i = 0; i < (int64_t)R * d; ++i) out[i] = 0.0;\n"
                            "    for (int32_t r = 0; r < R; ++r) lse[r] = 0.0;"),
    "tokens_empty_lse_zero": ("  if (ntoks == 0) { /* nothing to attend: the empty sum */\n"
                              "    for (int64_t i = 0; i < (int64_t)R * d; ++i) out[i] = 0.0;\n"
                              "    for (int32_t r = 0; r < R; ++r) lse[r] = -INFINITY;",
                              "  if (ntoks == 0) { /* nothing to attend: the empty sum */\n"
                              "    for (int64_t i = 0; i < (int64_t)R * d; ++i) out[i] = 0.0;\n"
                              "    for (int32_t r = 0; r < R; ++r) lse[r] = 0.0;"),
    "idx_dropped_relu": ("const double relu = dot > 0.0 ? dot : 0.0;", "const double relu = dot;"),
    "idx_gate_inside_relu": ("x += (double)w[h] * relu;",
                             "x += (double)w[h] * dot > 0.0 ? (double)w[h] * dot : 0.0;"),
    "idx_wrong_head_weight": ("x += (double)w[h] * relu;", "x += (double)w[(h + 1) % n_h] * relu;"),
    "idx_k_reversed_dims": ("bf16_to_f64(K[s * c + i])", "bf16_to_f64(K[s * c + (c - 1 - i)])"),
    "recall_strict_threshold": ("if (xl >= 0.0) recalled = 1;", "if (xl > 0.0) recalled = 1;"),
    "recall_first_layer_only": ("for (int32_t l = 0; l < L; ++l) {\n      const double xl",
                                "for (int32_t l = 0; l < 1; ++l) {\n      const double xl"),
    "recall_ranks_first_layer": ("if (xl > best) best = xl;", "if (xl > best && l < 0) best = xl;"),
    "recall_bound_ignored": ("  if (m > kmax) {", "  if (m > n) {"),
    "tokens_dropped_scale": ("      w[i] = dot * scale;", "      w[i] = dot;"),
    "tokens_v_wrong_token": ("acc += w[i] * bf16_to_f64(Vh[toks[i] * d + e]);",
                             "acc += w[i] * bf16_to_f64(Vh[toks[ntoks - 1 - i] * d + e]);"),
    "two_level_native_by_position": ("      v[j].s = native[recalled[j]];", "      v[j].s = native[j];"),
    "two_level_budget_ignored": ("    if (m > k2) {", "    if (m > n_hist) {"),
    "two_level_window_short": ("  for (int64_t c = w0; c < n_total; ++c)", "  for (int64_t c = w0 + 1; c < n_total; ++c)"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique/present"
    path = tmp_path / "mutant.c"
    path.write_text(src.replace(old, new))
    so = tmp_path / "libmutant.so"
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", str(path), "-o", str(so), "-lm"])
    saved = oracle._lib
    oracle._lib = oracle.bind(str(so))
    failed = []
    try:
        for pin in P.ALL_PINS:
            try:
                pin()
            except AssertionError:
                failed.append(pin.__name__)
            except ValueError:
                failed.append(pin.__name__)
    finally:
        oracle._lib = saved
    assert failed, f"no pin catches mutant {name}"
