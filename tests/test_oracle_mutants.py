"""Plausible mistakes planted in a copy of the oracle's C source must each fail
at least one pin.  This checks the pins, not the oracle: a pin set that a
dropped term, a wrong sign, index or grouping could slip through would be
useless.  Every mutation keeps memory accesses in bounds."""
import os

import pytest

import oracle as oracle_mod
from oracle_pins import ALL_PINS

SOURCES = oracle_mod.SOURCES

MUTANTS = {
    "scale_1_over_D": ("scale = 1.0 / sqrt((double)D);", "scale = 1.0 / (double)D;"),
    "gqa_modulo_grouping": ("for (int h = g * G; h < (g + 1) * G; ++h)",
                            "for (int h = g; h < Hq; h += Hkv)"),
    "no_max_subtraction": ("if (logit[t] > mx) mx = logit[t];", "mx = 0.0;"),
    "no_normalisation": ("imp[t] += exp(logit[t] - mx) / z;", "imp[t] += exp(logit[t] - mx);"),
    "reversed_query_channels": ("widen(q, dtype, qbase + d)", "widen(q, dtype, qbase + (D - 1 - d))"),
    "dropped_last_channel": ("for (int d = 0; d < D; ++d)", "for (int d = 0; d < D - 1; ++d)"),
    "ties_to_later_index": ("return (a->index < b->index) ? -1 : (a->index > b->index);",
                            "return (a->index > b->index) ? -1 : (a->index < b->index);"),
    "ascending_scores": ("if (a->key > b->key) return -1;\n    if (a->key < b->key) return 1;",
                         "if (a->key < b->key) return -1;\n    if (a->key > b->key) return 1;"),
    "output_not_in_source_order": ("qsort(out, (size_t)keep, sizeof(int32_t), ascending_i32);", ""),
    "nan_ranks_highest": ("return a->is_nan ? 1 : -1;", "return a->is_nan ? -1 : 1;"),
    "budget_floor": ("? nearest : ceil(x);", "? nearest : floor(x);"),
    "budget_no_noise_guard": ("(fabs(x - nearest) <= tol) ? nearest : ceil(x)", "ceil(x)"),
    "compact_sender_major": ("((((size_t)l * Hkv + g) * S + s) * (size_t)keep + j) * row",
                             "((((size_t)s * L + l) * Hkv + g) * (size_t)keep + j) * row"),
    "lse_off_by_log": ("= mx + log(z);", "= mx + log(z + 1.0);"),
    "bf16_wrong_shift": ("(uint32_t)((const uint16_t*)base)[i] << 16",
                         "(uint32_t)((const uint16_t*)base)[i] << 15"),
    "softmax_over_rows_sum_exp_only_first": ("for (int64_t t = 0; t < T; ++t) z += exp(logit[t] - mx);",
                                             "for (int64_t t = 0; t < 1; ++t) z += exp(logit[t] - mx);"),
    # position-level score (message.c)
    "numerator_mean_before_pool": (
        "pool_max(b + (size_t)r * T, T, pool_width, pooled);\n          for (int64_t t = 0; t < T; ++t) {",
        "pool_max(b, T, 1, pooled);\n          for (int64_t t = 0; t < T; ++t) {"),
    "denominator_pool_before_mean": ("pool_max(mean_b, T, pool_width, pooled);",
                                     "pool_max(mean_b, T, 1, pooled);"),
    "correction_without_inverse_power": ("c = pow(num[t] / den[t], 1.0 / (p - 1.0));",
                                         "c = num[t] / den[t];"),
    "score_linear_in_correction": ("score[o] = qpool[t] * pow(c, alpha);", "score[o] = qpool[t] * c;"),
    "pool_window_not_centred": ("int64_t lo = t - half < 0 ? 0 : t - half;", "int64_t lo = t;"),
    "pool_width_five": ("const int64_t half = (w - 1) / 2;", "const int64_t half = w > 1 ? 2 : 0;"),
    "q_mean_over_layers": ("q_pre[t] += a[(size_t)r * T + t] / ((double)m * Hq);",
                           "q_pre[t] += a[(size_t)r * T + t] / ((double)m * Hq * L);"),
    "q_not_pooled": ("pool_max(q_pre, T, pool_width, qpool);", "pool_max(q_pre, T, 1, qpool);"),
    "correction_zero_when_both_vanish": ("        c = 1.0;\n", "        c = 0.0;\n"),
    "b_modulo_grouping": ("attention_rows(q, k, dtype, L, Hq, Hkv, D, m, T, scale, s, l, h, g, a);",
                          "attention_rows(q, k, dtype, L, Hq, Hkv, D, m, T, scale, s, l, "
                          "(h - g * G) * Hkv + g, g, a);"),
    "p_inf_sums_instead_of_max": ("if (pooled[t] > num[t]) num[t] = pooled[t];", "num[t] += pooled[t] / m;"),
    # budgets and span rule (message.c)
    "fanout_budget_floor": ("return (T + r - 1) / r;", "return T / r;"),
    "chain_relative_drops_inherited": ("if (relative) return T_old + (T_new + r - 1) / r;",
                                       "if (relative) return (T_old + T_new + r - 1) / r;"),
    "spans_ties_to_later": ("return (a->span < b->span) ? -1 : (a->span > b->span);",
                            "return (a->span > b->span) ? -1 : (a->span < b->span);"),
    "spans_rank_by_sum": ("spans[j].key = sum / (double)(hi - lo);", "spans[j].key = sum;"),
    "first_position_keeps_its_score": ("  s[0] = mx;\n", "\n"),
    "latents_not_forced": ("  for (int64_t t = T - n_latent; t < T; ++t)\n    if (!sel[t]) {",
                           "  for (int64_t t = T; t < T; ++t)\n    if (!sel[t]) {"),
    "partial_interval_left_first": ("int64_t right = top + d, left = top - d;",
                                    "int64_t right = top - d, left = top + d;"),
    "partial_interval_from_span_start": ("    int64_t top = lo;\n    for (int64_t t = lo + 1; t < hi; ++t)\n      if (s[t] > s[top]) top = t;",
                                         "    int64_t top = lo;"),
    "partial_span_skipped": ("    /* the span does not fit: an interval around its top position */",
                             "    continue;"),
    "gather_rows_wrong_sender": ("(const char*)rows + ((size_t)s * T + t) * row_bytes",
                                 "(const char*)rows + ((size_t)0 * T + t) * row_bytes"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    before, after = MUTANTS[name]
    texts = [open(src).read() for src in SOURCES]
    hits = [t.count(before) for t in texts]
    # an anchor found in both sources plants the same mistake in both
    assert sum(hits) >= 1 and max(hits) == 1, f"mutation anchor for {name} not found exactly once"
    paths = []
    for src, text, n in zip(SOURCES, texts, hits):
        path = tmp_path / os.path.basename(src)
        path.write_text(text.replace(before, after) if n else text)
        paths.append(str(path))
    # the mutant includes oracle.h from the oracle's directory
    so = oracle_mod.build(srcs=paths, out=str(tmp_path / f"lib_{name}.so"))
    orc = oracle_mod.Oracle(so)
    failures = []
    for pin in ALL_PINS:
        try:
            pin(orc)
        except (AssertionError, RuntimeError, ValueError, FloatingPointError):
            failures.append(pin.__name__)
    assert failures, f"mutant {name} passed every pin"
