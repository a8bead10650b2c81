"""The pins must catch plausible mistakes in the oracle.

Each case copies the oracle's C source to a temporary directory, plants one
mistake (a dropped term, a wrong sign or index, a transposed operand, a
non-strict threshold, ...), compiles the copy and runs the pin checks of
test_oracle_pins against it: at least one must fail.  Nothing here touches
the real oracle or any GPU.
"""
import os
import shutil

import pytest

import oracle
import test_oracle_pins as pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "fork_oracle.c")
HDR = os.path.join(os.path.dirname(oracle.__file__), "fork_oracle.h")

MUTATIONS = {
    "argmax_tie_highest": ("if (z[v] > z[a]) a = v;", "if (z[v] >= z[a]) a = v;"),
    "drop_first_product": ("for (int64_t j = 0; j < d; ++j)", "for (int64_t j = 1; j < d; ++j)"),
    "transposed_weight": ("widen(W, dtype, v * d + j)", "widen(W, dtype, j * V + v)"),
    "no_max_shift": ("sum += exp(z[v] - zmax);", "sum += exp(z[v]);"),
    "entropy_sign": ("h -= exp(lq) * lq;", "h += exp(lq) * lq;"),
    "entropy_drops_norm": ("double lq = z[v] - log_norm;", "double lq = z[v] - z[0];"),
    "logp_drops_logit": ("*logp = z[a] - log_norm;", "*logp = -log_norm;"),
    "conf_unnormalised": ("*conf = exp(z[a] - log_norm);", "*conf = exp(z[a] - zmax);"),
    "threshold_not_strict": ("conf[base + k] > lambda", "conf[base + k] >= lambda"),
    "no_block_limit": ("const int32_t e = s + block_len < L ? s + block_len : L;",
                       "const int32_t e = L;"),
    "rightmost_fallback": ("if (rule == ORACLE_RULE_LEFTMOST) break;",
                           "if (rule == ORACLE_RULE_LEFTMOST) continue;"),
    "fallback_flag_swapped": ("fallback[b] = 1;\n    } else {\n      fallback[b] = 0;",
                              "fallback[b] = 0;\n    } else {\n      fallback[b] = 1;"),
    "fast_tie_highest": ("(cand < best) : (cand > best);", "(cand <= best) : (cand >= best);"),
    "minconf_as_maxconf": ("rule == ORACLE_RULE_MINCONF ? (cand < best)", "rule == ORACLE_RULE_MINCONF ? (cand > best)"),
    "maxent_reads_conf": ("const double* key = rule == ORACLE_RULE_MAXENT ? entropy : conf;",
                          "const double* key = conf;"),
    "random_off_by_one": ("if (mask[base + k] && j-- == 0) return k;", "if (mask[base + k] && --j == 0) return k;"),
    "random_rounds_up": ("int32_t j = (int32_t)prod;", "int32_t j = (int32_t)(prod + 0.5f);"),
    "no_skip_forward": ("s += block_len;", "break;"),
    "philox_multiplier": ("0xD2511F53u", "0xD2511F55u"),
    "philox_no_key_bump": ("k[1] += 0xBB67AE85u;", ""),
    "philox_words_swapped": ("c[0] = n0;\n  c[1] = lo1;", "c[0] = lo1;\n  c[1] = n0;"),
    "draw_counter_layout": ("{(uint32_t)(v / 4), (uint32_t)row, counter, 0u}",
                            "{(uint32_t)(v / 4), counter, (uint32_t)row, 0u}"),
    "gumbel_sign": ("z[v] / tau - log(oracle_exp_draw(", "z[v] / tau + log(oracle_exp_draw("),
    "temperature_multiplies": ("z[v] / tau - log(", "z[v] * tau - log("),
    "sample_logq_drops_logit": ("const double log_q = z[a] - log_norm;",
                              "const double log_q = log_norm - log_norm;"),
    "keygap_stale_second": ("      second = best;\n      best = key;", "      best = key;"),
    "logprob_wrong_index": ("logp[e] = z[tokens[e]] - log_norm;", "logp[e] = z[e] - log_norm;"),
    "grpo_std_divisor": ("sqrt(var / G)", "sqrt(var / (G - 1))"),
    "grpo_max_not_min": ("const double tm = a < b ? a : b;", "const double tm = a > b ? a : b;"),
    "grpo_clip_lower_bound": ("rho < 1.0 - eps ? 1.0 - eps", "rho < 1.0 - eps ? 1.0 + eps"),
    "grpo_no_skip": ("const int skip = !(sd > 0.0);", "const int skip = 0;"),
    "grpo_rollout_sum": ("nF > 0 ? acc / nF : 0.0", "nF > 0 ? acc : 0.0"),
    "grpo_mean_over_all_groups": ("kept > 0 ? total / kept : 0.0", "n_groups > 0 ? total / n_groups : 0.0"),
    "top_entropy_tie_highest": ("(h[q] == h[p] && q < p)", "(h[q] == h[p] && q > p)"),
    "top_entropy_lowest": ("if (h[q] > h[p] ||", "if (h[q] < h[p] ||"),
}


def _checks(orc):
    """Run the pin suite's checks against one oracle build; returns the
    number of failing checks."""
    calls = [
        lambda: pins.test_stats_match_dense_brute_force(orc, 1, 7, 16, 33, "f32", 1.0),
        lambda: pins.test_stats_match_dense_brute_force(orc, 3, 9, 40, 257, "bf16", 3.0),
        lambda: pins.test_uniform_closed_form(orc, 1024),
        lambda: pins.test_k_way_tie_closed_form(orc, 7, 0),
        lambda: pins.test_two_level_closed_form(orc, 3.0, 0.0, 10),
        lambda: pins.test_shift_invariance(orc),
        lambda: pins.test_select_hand_worked_fixture(orc),
        lambda: pins.test_lambda_at_least_one_is_autoregressive(orc, 1.0),
        lambda: pins.test_lambda_zero_commits_whole_blocks(orc),
        lambda: pins.test_select_invariants(orc, 0, 0.8),
        lambda: pins.test_fork_vs_fast_differential(orc, 0),
        lambda: pins.test_fast_fallback_tie_takes_lowest_position(orc),
        lambda: pins.test_fallback_ablations_hand_worked(orc),
        lambda: pins.test_fallback_ablation_properties(orc, 0),
        lambda: pins.test_philox_known_answers(orc),
        lambda: pins.test_exp_draw_layout_and_law(orc),
        lambda: pins.test_sample_frequencies_follow_tempered_softmax(orc, 0.5),
        lambda: pins.test_sample_low_temperature_is_greedy(orc),
        lambda: pins.test_sample_brute_force_keys(orc),
        lambda: pins.test_token_logprob_brute_force(orc),
        lambda: pins.test_grpo_hand_worked_fixture(orc),
        lambda: pins.test_grpo_invariants(orc, 0),
        lambda: pins.test_top_entropy_hand_worked(orc),
        lambda: pins.test_top_entropy_matches_sort(orc, 52),
    ]
    failed = 0
    for c in calls:
        try:
            c()
        except (AssertionError, ValueError, FloatingPointError, IndexError):
            failed += 1
    return failed


def test_unmutated_copy_passes(tmp_path):
    shutil.copy(HDR, tmp_path)
    src = tmp_path / "fork_oracle.c"
    shutil.copy(SRC, src)
    lib = oracle.build(force=True, src=str(src), out=str(tmp_path / "lib.so"))
    assert _checks(oracle.Oracle(lib)) == 0


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(tmp_path, name):
    old, new = MUTATIONS[name]
    text = open(SRC).read()
    assert text.count(old) == 1, "mutation anchor must occur exactly once"
    shutil.copy(HDR, tmp_path)
    src = tmp_path / "fork_oracle.c"
    src.write_text(text.replace(old, new))
    lib = oracle.build(force=True, src=str(src), out=str(tmp_path / ("%s.so" % name)))
    assert _checks(oracle.Oracle(lib)) > 0, "planted mistake %r went unnoticed" % name
