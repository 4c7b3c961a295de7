"""Plausible mistakes planted in a copy of the oracle's C source must each fail
at least one pin.  This checks the pins, not the oracle: a pin set that a
dropped term, a wrong sign, index or grouping could slip through would be
useless.  Every mutation keeps memory accesses in bounds."""
import os

import pytest

import oracle as oracle_mod
from oracle_pins import ALL_PINS

SRC = os.path.join(os.path.dirname(oracle_mod.__file__), "oracle.c")

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
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    before, after = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(before) == 1, f"mutation anchor for {name} not found exactly once"
    path = tmp_path / "mutant.c"
    path.write_text(src.replace(before, after))
    # the mutant includes oracle.h from the oracle's directory
    so = oracle_mod.build(src=str(path), out=str(tmp_path / f"lib_{name}.so"))
    orc = oracle_mod.Oracle(so)
    failures = []
    for pin in ALL_PINS:
        try:
            pin(orc)
        except (AssertionError, RuntimeError, ValueError, FloatingPointError):
            failures.append(pin.__name__)
    assert failures, f"mutant {name} passed every pin"
