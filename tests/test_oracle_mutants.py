"""Planted mistakes in the oracle must be caught by its pins.

Each mutant is a one-line textual change to ``oracle/lsa_oracle.c`` -- a
reversed tie-break, a dropped scale, a wrong sign, a wrong token or dimension
index, a dropped term -- compiled on the CPU into a throw-away library, or to
the plain-Python parts of ``oracle/__init__.py`` (the two-level window and the
host tier's residency plan), executed into a throw-away module.  The
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
    "top_p_strict_mass": ("if ((double)(p_den - p_num) * head >= (double)p_num * tail[j + 1]) size = j + 1;",
                          "if ((double)(p_den - p_num) * head > (double)p_num * tail[j + 1]) size = j + 1;"),
    "top_p_tail_includes_entry": ("if ((double)(p_den - p_num) * head >= (double)p_num * tail[j + 1]) size = j + 1;",
                                  "if ((double)(p_den - p_num) * head >= (double)p_num * tail[j]) size = j + 1;"),
    "top_p_head_for_total": ("if ((double)(p_den - p_num) * head >= (double)p_num * tail[j + 1]) size = j + 1;",
                             "if ((double)p_den * head >= (double)p_num * tail[j + 1]) size = j + 1;"),
    "top_p_tie_reversed": ("  return (x->c > y->c) - (x->c < y->c);\n}\n\n/*\n * Top-p set",
                           "  return (x->c < y->c) - (x->c > y->c);\n}\n\n/*\n * Top-p set"),
    "top_p_least_probable_first": ("  if (x->s > y->s) return -1;\n  if (x->s < y->s) return 1;\n"
                                   "  return (x->c > y->c) - (x->c < y->c);\n}\n\n/*\n * Top-p set",
                                   "  if (x->s > y->s) return 1;\n  if (x->s < y->s) return -1;\n"
                                   "  return (x->c > y->c) - (x->c < y->c);\n}\n\n/*\n * Top-p set"),
    "top_p_tail_not_summed": ("for (int64_t j = n - 1; j >= 0; --j) tail[j] = tail[j + 1] + w[j];",
                              "for (int64_t j = n - 1; j >= 0; --j) tail[j] = w[j];"),
    "top_p_logits_doubled": ("for (int64_t j = 0; j < n; ++j) w[j] = exp((double)v[j].s - m);",
                                       "for (int64_t j = 0; j < n; ++j) w[j] = exp(2.0 * ((double)v[j].s - m));"),
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


# Mutants of the plain-Python parts of the oracle (oracle/__init__.py): the
# window of the two-level path and the host tier's residency plan.
PY_MUTANTS = {
    "window_whole_chunks_only": ("        holds_recent = hi > ctx_tokens - window_tokens\n",
                                 "        holds_recent = lo >= ctx_tokens - window_tokens\n"),
    "window_partial_not_resident": ("        in_window.append(holds_recent or partial)\n",
                                    "        in_window.append(holds_recent)\n"),
    "window_tail_off_by_one": ("    return w0, n_total, ctx_tokens - (n_total - 1) * chunk\n",
                               "    return w0, n_total, ctx_tokens - n_total * chunk + chunk - 1\n"),
    "tier_free_slots_descending": ("    free = [s for s in range(len(owner)) if s not in protected]\n",
                                   "    free = [s for s in reversed(range(len(owner))) if s not in protected]\n"),
    "tier_previous_set_unprotected": ("    protected = set(old_slots) | {where[c] for c in kept if c in where}\n",
                                      "    protected = {where[c] for c in kept if c in where}\n"),
    "tier_missing_descending": ("    fetch = list(zip(missing, free))\n", "    fetch = list(zip(reversed(missing), free))\n"),
    "tier_resident_recopied": ("    missing = [c for c in kept if c not in where]\n", "    missing = list(kept)\n"),
}


@pytest.mark.parametrize("name", sorted(PY_MUTANTS))
def test_python_mutant_is_caught(name):
    import types
    old, new = PY_MUTANTS[name]
    path = os.path.join(os.path.dirname(oracle.__file__), "__init__.py")
    src = open(path).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique/present"
    mod = types.ModuleType("oracle_mutant")
    mod.__file__ = path
    exec(compile(src.replace(old, new), path, "exec"), mod.__dict__)
    saved = {f: getattr(oracle, f) for f in ("window", "tier_plan")}
    for f in saved:
        setattr(oracle, f, getattr(mod, f))
    failed = []
    try:
        for pin in P.ALL_PINS:
            try:
                pin()
            except (AssertionError, ValueError, KeyError):
                failed.append(pin.__name__)
    finally:
        for f, fn in saved.items():
            setattr(oracle, f, fn)
    assert failed, f"no pin catches mutant {name}"


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
