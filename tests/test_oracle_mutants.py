"""The pins must catch plausible mistakes in the oracle.

Each case plants one mistake (a dropped term, a wrong index, a flipped
comparison, a wrong mask) in a temporary copy of the oracle's C source, builds
it with gcc, swaps it in for the real library and checks that at least one
pin of ``test_oracle_pins`` fails on it. CPU only.
"""
import ctypes
import os
import subprocess

import pytest

import oracle
from oracle import build as obuild

from . import test_oracle_pins as P

MUTANTS = [
    ("diagonal_not_antidiagonal", "(size_t)(R * S + S - 1 - t) * D", "(size_t)(R * S + t) * D"),
    ("key_subrow_reversed", "(size_t)(c * S + t) * D", "(size_t)(c * S + S - 1 - t) * D"),
    ("score_scale_drops_stride", "1.0 / (sqrt((double)D) * (double)S)", "1.0 / sqrt((double)D)"),
    ("score_block_causal_mask", "d->causal ? R + 1 : NR", "d->causal ? (b + 1) * nr : NR"),
    ("score_no_row_mean", "row[j] /= (double)nr;", "row[j] /= 1.0;"),
    ("score_wrong_block_of_column", "row[c / nr] +=", "row[(c % NB)] +="),
    ("gqa_interleaved_groups", "hh / (d->hq / d->hkv)", "hh % d->hkv"),
    ("select_strict_threshold", "if (cum >= target) break;", "if (cum > target) break;"),
    ("select_floor_target", "(uint64_t)ceil(prod)", "(uint64_t)floor(prod)"),
    ("select_ties_high_index_first", "return x->j < y->j ? -1 : (x->j > y->j);",
     "return x->j > y->j ? -1 : (x->j < y->j);"),
    ("select_ignores_tau_one", "if (tau >= 1.0f) {", "if (tau >= 2.0f) {"),
    ("attn_scale_wrong", "const double scale = 1.0 / sqrt((double)D);\n    double m = -INFINITY;\n    for (int t = 0; t < nk; ++t)",
     "const double scale = 1.0 / (double)D;\n    double m = -INFINITY;\n    for (int t = 0; t < nk; ++t)"),
    ("sparse_causal_strict", "if (!d->causal || kk <= qi) keys[nk++] = kk;",
     "if (!d->causal || kk < qi || kk == 0) keys[nk++] = kk;"),
    ("dense_causal_off_by_one", "const int nk = d->causal ? qi + 1 : L;\n            for (int kk = 0; kk < nk; ++kk) keys[kk] = kk;",
     "const int nk = d->causal ? (qi > 0 ? qi : 1) : L;\n            for (int kk = 0; kk < nk; ++kk) keys[kk] = kk;"),
    ("attn_value_row_wrong", "const uint16_t *vr = V + (size_t)keys[t] * D;",
     "const uint16_t *vr = V + (size_t)(nk - 1 - t) * D;"),
    ("pattern_ignores_pairing", "(size_t)(R * S + qsub[t]) * D", "(size_t)(R * S + t) * D"),
    ("pattern_pairing_reversed", "(size_t)(R * S + qsub[t]) * D",
     "(size_t)(R * S + qsub[S - 1 - t]) * D"),
    ("topk_takes_the_tail", "for (int t = 0; t < k; ++t) out[t] = c[t].j;",
     "for (int t = 0; t < k; ++t) out[t] = c[m - 1 - t].j;"),
    ("topk_output_unsorted", "qsort(out, (size_t)k, sizeof(int32_t), int_cmp);\n        cnt[i] = k;",
     "cnt[i] = k;"),
    ("topk_off_by_one", "for (int t = 0; t < k; ++t) out[t] = c[t].j;",
     "for (int t = 0; t < k; ++t) out[t] = c[t + (t + 1 < m)].j;"),
    ("ratio_rounds_up", "floor((double)ratio_row[i] * (double)m + 0.5)",
     "ceil((double)ratio_row[i] * (double)m)"),
    ("ratio_rounds_down", "floor((double)ratio_row[i] * (double)m + 0.5)",
     "floor((double)ratio_row[i] * (double)m)"),
]

PINS = [
    lambda: P.test_score_equals_antidiagonal_index_walk(4, True, 16),
    lambda: P.test_score_equals_antidiagonal_index_walk(8, False, 128),
    P.test_score_walk_on_clustered_inputs,
    lambda: P.test_stride_one_is_exact_block_mass(True),
    P.test_score_rows_sum_to_one_and_causal_zeros,
    lambda: P.test_zero_query_closed_form(4),
    lambda: P.test_select_matches_subset_enumeration(3, True),
    lambda: P.test_select_matches_subset_enumeration(1, False),
    P.test_select_small_integer_masses_match_subset_enumeration,
    P.test_select_tau_one_takes_every_candidate_even_zero_mass,
    P.test_select_monotone_in_tau_and_ties_prefer_low_index,
    lambda: P.test_dense_matches_torch_sdpa(True),
    lambda: P.test_sparse_equals_block_masked_attention(True),
    P.test_zero_query_attention_is_running_mean_of_values,
    lambda: P.test_score_pattern_equals_masked_index_walk("random", 4, True),
    lambda: P.test_score_pattern_equals_masked_index_walk("diagonal", 8, False),
    lambda: P.test_topk_is_the_upper_set_of_the_selection_order(False),
    lambda: P.test_topk_is_the_upper_set_of_the_selection_order(True),
    P.test_topk_sets_nest_and_match_threshold_selection_at_its_count,
    P.test_topk_brute_force_mass_is_maximal,
] + [lambda a=a: P.test_ratio_block_count_rounds_to_nearest(*a) for a in [
    (0.5, 3, 2), (0.27, 100, 27), (0.7, 10, 7), (0.01, 3, 1), (2.0, 4, 4)]]


def _build_mutant(tmp_path, name, old, new):
    src = open(obuild.SRC).read()
    # the site is its first occurrence (the scoring pattern variant repeats a
    # few lines of the Algorithm 1 scoring, which comes first in the file)
    assert src.count(old) >= 1, f"mutation site absent: {name}"
    path = tmp_path / f"{name}.c"
    path.write_text(src.replace(old, new, 1))
    lib = tmp_path / f"lib{name}.so"
    subprocess.run(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                    "-ffp-contract=off", str(path), "-o", str(lib), "-lm"], check=True)
    return str(lib)


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_mutant(tmp_path, name, old, new):
    lib_path = _build_mutant(tmp_path, name, old, new)
    real = oracle.lib()
    L = ctypes.CDLL(lib_path)
    for f in ("oracle_score_rows", "oracle_select_rows", "oracle_sparse_attn_rows",
              "oracle_dense_attn_rows", "oracle_block_mass_rows", "oracle_select_topk_rows",
              "oracle_select_ratio_rows", "oracle_score_pattern_rows"):
        getattr(L, f).argtypes = getattr(real, f).argtypes
    L.oracle_num_threads.restype = ctypes.c_int
    caught = []
    oracle._LIB = L
    try:
        for pin in PINS:
            try:
                pin()
            except (AssertionError, ValueError, FloatingPointError):
                caught.append(pin)
                break
    finally:
        oracle._LIB = real
    assert caught, f"no pin caught mutant {name}"


def test_real_oracle_passes_the_same_pins():
    for pin in PINS:
        pin()
    assert os.path.exists(obuild.LIB)
