"""The pins must catch plausible mistakes in the oracle.

Each case plants one mistake (a flipped comparison, a dropped term, a transposed operand, a wrong
tie rule ...) in a private copy of the oracle source, builds it with gcc on the CPU, points the
oracle wrapper at that build and checks that at least one pin fails.  The real oracle is restored
afterwards."""
from __future__ import annotations

import os
import subprocess
import tempfile

import numpy as np
import pytest

import oracle
from tests import test_oracle_gbdt as gb
from tests import test_oracle_pins as pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "harl_oracle.c")

MUTANTS = {
    "split_not_strict": ("(v < threshold[n])", "(v <= threshold[n])",
                         [(pins.test_threshold_ties_and_missing, dict(thr=np.float32(1.5), dl=0))]),
    "default_dir_swapped": ("default_left[n] ? left[n] : right[n]", "default_left[n] ? right[n] : left[n]",
                            [(pins.test_all_missing_row_follows_default_bits, {})]),
    "missing_not_detected": ("if (isnan(v))", "if (0)",
                             [(pins.test_threshold_ties_and_missing, dict(thr=np.float32(1.5), dl=1))]),
    "first_tree_dropped": ("for (int32_t t = 0; t < n_trees; ++t)", "for (int32_t t = 1; t < n_trees; ++t)",
                           [(pins.test_tree_sums_match_path_predicates, dict(p_nan=0.0, depth=3))]),
    "program_keeps_last_stmt": ("acc += s;", "acc = s;",
                                [(pins.test_leafless_root_and_constant_leaves_closed_form, {})]),
    "base_score_ignored": ("double acc = base_score, sc", "double acc = 0.0, sc",
                           [(pins.test_base_score_and_empty_programs, {})]),
    "layer2_bias_dropped": ("double acc = b2[i];", "double acc = 0.0;",
                            [(pins.test_policy_matches_numpy_matmul, dict(dtype="f32"))]),
    "relu_missing": ("acc = acc > 0.0 ? acc : 0.0;\n                    h1[i]", "h1[i]",
                     [(pins.test_policy_matches_numpy_matmul, dict(dtype="f32"))]),
    "w2_transposed": ("load_val(w2, dtype, (int64_t)i * H1 + j)", "load_val(w2, dtype, (int64_t)j * H2 + i)",
                      [(pins.test_policy_matches_numpy_matmul, dict(dtype="f32"))]),
    "argmax_last_tie": ("if (acc > z[best]) best = i;", "if (acc >= z[best]) best = i;",
                        [(pins.test_policy_exact_integer_variant, dict(dtype="f32"))]),
    "bf16_rounding_skipped": ("h2[i] = dtype == 1 ? round_to_bf16(acc) : acc;", "h2[i] = acc;",
                              [(pins.test_policy_matches_numpy_matmul, dict(dtype="bf16"))]),
    "bf16_ties_away": ("(frac == 0.5 && fmod(fl, 2.0) != 0.0)", "(frac == 0.5)",
                       [(pins.test_bf16_rounding_rule, {})]),
    "softmax_unnormalised": ("exp(z[i] - m) / sum", "exp(z[i] - m)",
                             [(pins.test_softmax_invariants, {})]),
    "topk_index_desc": ("if (a->index < b->index) return -1;\n    if (a->index > b->index) return 1;",
                        "if (a->index < b->index) return 1;\n    if (a->index > b->index) return -1;",
                        [(pins.test_topk_matches_lexsort, {})]),
    "nan_ranked_first": ("if (an != bn) return an ? 1 : -1;", "if (an != bn) return an ? -1 : 1;",
                         [(pins.test_topk_special_cases, {})]),
    "merge_local_index": ("c[k + i].index = index_base + i;", "c[k + i].index = i;",
                          [(pins.test_merge_equals_topk_of_union_in_any_order, {})]),
    "reward_signed_denominator": ("fabs(c) > eps ? fabs(c) : eps", "c > eps ? c : eps",
                                  [(pins.test_reward_advantage_closed_forms, {})]),
    "reward_no_eps_floor": ("fabs(c) > eps ? fabs(c) : eps", "fabs(c)",
                            [(pins.test_reward_advantage_closed_forms, {})]),
    "advantage_discounts_prev": ("const double g = gamma * (double)v_next[i];",
                                 "const double g = gamma * (double)v_prev[i];",
                                 [(pins.test_reward_advantage_closed_forms, {})]),
    "advantage_value_sign": ("adv[i] = r + g - v;", "adv[i] = r + g + v;",
                             [(pins.test_reward_sign_and_critic_reductions, {})]),
    "eliminate_keeps_worst": ("keep[c[k].index] = 1;", "keep[c[n - 1 - k].index] = 1;",
                              [(pins.test_eliminate_special_cases, {})]),
    "eliminate_rank_order_out": ("if (keep[i]) keep_index[m++] = (int32_t)i;",
                                 "if (keep[i]) keep_index[m++] = (int32_t)i;\n    for (int64_t k = 0; k < n_keep; ++k) keep_index[k] = (int32_t)c[k].index;",
                                 [(pins.test_eliminate_ranking_properties_small, {})]),
    "philox_multipliers_swapped": ("(uint64_t)M0 * c[0], p1 = (uint64_t)M1 * c[2]",
                                   "(uint64_t)M1 * c[0], p1 = (uint64_t)M0 * c[2]",
                                   [(pins.test_philox_known_answers, {})]),
    "philox_key_bumped_first": ("if (round > 0) {\n            k[0] += W0;", "if (round >= 0) {\n            k[0] += W0;",
                                [(pins.test_philox_known_answers, {})]),
    "select_last_tie": ("if (key > best) {", "if (key >= best) {",
                        [(pins.test_greedy_select_is_per_segment_first_argmax, {})]),
    "gumbel_sign": ("return -log(-log(u));", "return log(-log(u));",
                    [(pins.test_sampling_frequencies_follow_the_softmax, {})]),
    "logp_unnormalised": ("logp[b * n_seg + s] = (double)z[pick] - m - log(sum);",
                          "logp[b * n_seg + s] = (double)z[pick] - m;",
                          [(pins.test_select_softmax_and_logp_identities, {})]),
    "segment_shifted": ("const int32_t lo = off[s], hi = off[s + 1];", "const int32_t lo = off[s], hi = off[s + 1] - (s == 0);",
                        [(pins.test_greedy_select_is_per_segment_first_argmax, {})]),
    "gbdt_bin_strict": ("if (cuts[f * cut_stride + i] <= v) ++c;", "if (cuts[f * cut_stride + i] < v) ++c;",
                        [(gb.test_bins_are_searchsorted_counts, {})]),
    "gbdt_threshold_next_cut": ("c->cuts[(int64_t)bf * c->cut_stride + bt - 1]", "c->cuts[(int64_t)bf * c->cut_stride + bt]",
                                [(gb.test_step_function_single_split_closed_form, {})]),
    "gbdt_lambda_dropped": ("return (G * G) / (H + lambda);", "return (G * G) / (H + 1e-300);",
                            [(gb.test_tree_matches_exact_brute_force, dict(seed=2, depth=2, p_nan=0.0, lam=0.5))]),
    "gbdt_leaf_sign": ("const float w = (float)(-(G / (H + c->lambda)) * c->eta);",
                       "const float w = (float)((G / (H + c->lambda)) * c->eta);",
                       [(gb.test_step_function_single_split_closed_form, {})]),
    "gbdt_eta_dropped": ("const float w = (float)(-(G / (H + c->lambda)) * c->eta);",
                         "const float w = (float)(-(G / (H + c->lambda)));",
                         [(gb.test_isolated_programs_closed_form, {})]),
    "gbdt_hessian_one": ("h[p] = (double)weight[p];", "h[p] = 1.0;", [(gb.test_isolated_programs_closed_form, {})]),
    "gbdt_base_ignored": ("double s = base_score;", "double s = 0.0;", [(gb.test_isolated_programs_closed_form, {})]),
    "gbdt_pack_mean": ("g[p] = (double)weight[p] * (s - (double)label[p]);",
                       "g[p] = (double)weight[p] * (s / (prog_ptr[p + 1] - prog_ptr[p] + (prog_ptr[p + 1] == prog_ptr[p])) - (double)label[p]);",
                       [(gb.test_isolated_programs_closed_form, {})]),
    "gbdt_missing_right_first": ("for (int dir = 1; dir >= 0; --dir)", "for (int dir = 0; dir <= 1; ++dir)",
                                 [(gb.test_step_function_single_split_closed_form, {})]),
    "gbdt_missing_not_routed": ("const int go_left = b == 255 ? bdir : b < bt;", "const int go_left = b < bt;",
                                [(gb.test_missing_rows_follow_the_learned_direction, {})]),
    "gbdt_tie_last_feature": ("if (!found || gain > best) {", "if (!found || gain >= best) {",
                              [(gb.test_ties_go_to_the_lowest_feature_and_threshold, {})]),
    "gbdt_parent_not_subtracted": ("(node_score(GL, HL, c->lambda) + node_score(GR, HR, c->lambda)) - parent",
                                   "(node_score(GL, HL, c->lambda) + node_score(GR, HR, c->lambda))",
                                   [(gb.test_gamma_prunes_at_the_best_gain, {})]),
    "gbdt_mcw_ignored": ("if (!(HL >= c->mcw) || !(HR >= c->mcw)) continue;", "",
                         [(gb.test_min_child_weight_blocks_light_children, {})]),
    "gbdt_exponent_off": ("return 62 - ceil_log2_i64(n > 0 ? n : 1) - E;", "return 62 - ceil_log2_i64(n > 0 ? n : 1) - E + 1;",
                          [(gb.test_fixed_point_exponent_rule, {})]),
    "gbdt_children_swapped": ("int rc = grow(c, 2 * k + 1, depth + 1, lr, nl);\n        if (rc == ORACLE_OK) rc = grow(c, 2 * k + 2, depth + 1, rr, nr);",
                              "int rc = grow(c, 2 * k + 1, depth + 1, rr, nr);\n        if (rc == ORACLE_OK) rc = grow(c, 2 * k + 2, depth + 1, lr, nl);",
                              [(gb.test_new_tree_scores_like_the_margin_update, {})]),
}


@pytest.fixture(scope="module")
def workdir():
    with tempfile.TemporaryDirectory(prefix="harl_mutants_") as d:
        yield d
    oracle.use_library(None)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_planted_mistake(name, workdir):
    old, new, checks = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, "mutation site must be unique: %r" % old
    path_c = os.path.join(workdir, name + ".c")
    path_so = os.path.join(workdir, name + ".so")
    with open(path_c, "w") as f:
        f.write(src.replace(old, new))
    subprocess.run(["gcc", *oracle.CFLAGS, path_c, "-o", path_so, "-lm"], check=True)
    oracle.use_library(path_so)
    try:
        caught = 0
        for fn, kw in checks:
            try:
                fn(**kw)
            except (AssertionError, ValueError):
                caught += 1
        assert caught > 0, "planted mistake %s passed every pin" % name
    finally:
        oracle.use_library(None)
