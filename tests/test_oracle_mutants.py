"""Plant plausible mistakes in a copy of the oracle (CPU only) and check that
the pins catch every one.  The planted copies are compiled into a temporary
directory; the real oracle is untouched."""

import pytest

import oracle_pins as pins
from oracle import build_library, load_library
from oracle.oracle import _SRC

# Pruning at t = 0 as well is not listed: every arm is still in its initial
# state then, all scores tie, and the prune cannot remove anything, so that
# change is equivalent rather than a mistake.  Nor is dropping the action-space
# test from the argmax: arms outside the space score -inf, below any arm inside.
MUTANTS = {
    "eq3_dropped_outer_product": ("A[p * d + q] += x[p] * x[q];", "A[p * d + q] += x[p] * x[p];"),
    "eq4_wrong_sign": ("b[p] += r * x[p];", "b[p] -= r * x[p];"),
    "eq5_transposed_index": ("s += Ainv[p * d + q] * b[q];", "s += Ainv[p * d + q] * b[p];"),
    "score_wrong_operand": ("row += Ainv[p * d + q] * xi[q];", "row += Ainv[p * d + q] * xi[p];"),
    "lcb_wrong_sign": ("L[k] = greedy ? m : m - alpha * w;", "L[k] = greedy ? m : m + alpha * w;"),
    "ties_to_highest_index": ("(best < 0 || U[k] > U[best])", "(best < 0 || U[k] >= U[best])"),
    "prune_non_strict": ("if (act[k] && U[k] < lstar) kp[k] = 0;",
                         "if (act[k] && U[k] <= lstar) kp[k] = 0;"),
    "prune_period_off_by_one": ("(t % o->period) == 0", "((t + 1) % o->period) == 0"),
    "alpha_schedule_no_plus_one": ("sqrt((double)t + 1.0)", "sqrt((double)t + 2.0)"),
    "init_inverse_not_scaled": ("o->Ainv[(k * d + r) * d + r] = 1.0 / lambda;",
                                "o->Ainv[(k * d + r) * d + r] = lambda;"),
    "gauss_jordan_sign": ("W[r][c] -= f * W[col][c];", "W[r][c] += f * W[col][c];"),
    "update_wrong_arm": ("update_arm(o, i, a, o->xprev", "update_arm(o, i, (a + 1) % o->K, o->xprev"),
    "update_uses_current_context": ("update_arm(o, i, a, o->xprev + (size_t)i * o->d, r[i]);",
                                    "update_arm(o, i, a, o->xprev, r[i]);"),
    "width_without_root": ("double w = sqrt(quad > 0.0 ? quad : 0.0);",
                           "double w = quad > 0.0 ? quad : 0.0;"),
    "extreme_threshold_sign": ("double m = mean[k] - o->ext_thr;", "double m = mean[k] + o->ext_thr;"),
    "extreme_round_limit_inclusive": ("t < o->ext_rounds", "t <= o->ext_rounds"),
    "extreme_min_samples_off_by_one": ("n[k] >= o->ext_min_n", "n[k] > o->ext_min_n"),
    "historical_variance_not_rooted": ("double sigma = sqrt(var / q);", "double sigma = var / q;"),
    "historical_min_arms_ignored": ("if (q >= o->hist_min_arms && q > 0)", "if (q > 0)"),
    "historical_gap_reversed": ("double m = o->hist_kappa * sigma - (best - mean[k]);",
                                "double m = o->hist_kappa * sigma - (mean[k] - best);"),
    "cascade_prunes_upwards": ("for (int k = 0; k < kstar; ++k) gone[k] = 1;",
                               "for (int k = kstar + 1; k < K; ++k) gone[k] = 1;"),
    "cascade_threshold_inclusive": ("if (gone[k] && k < o->cascade_k) kstar = k;",
                                    "if (gone[k] && k <= o->cascade_k) kstar = k;"),
    "keep_one_worst_mean": ("(n[keep] == 0 || mean[k] > mean[keep])", "(n[keep] == 0 || mean[k] < mean[keep])"),
    "reward_sum_not_kept": ("    o->rsum[ik] += r;", "    o->rsum[ik] += 0.0 * r;"),
    "ph_drift_sign": ("p->up += (r - rbar) - o->ph_delta;", "p->up += (r - rbar) + o->ph_delta;"),
    "ph_minimum_not_tracked": ("if (p->up < p->up_min) p->up_min = p->up;", "p->up_min = p->up;"),
    "ph_no_restart": ("        memset(p, 0, sizeof(*p));\n", ""),
    "ph_mean_before_reward": ("const double rbar = p->sum / p->n;",
                              "const double rbar = p->n > 1.0 ? (p->sum - r) / (p->n - 1.0) : 0.0;"),
    "ph_one_sided": ("const double stat = fmax(p->up - p->up_min, p->dn - p->dn_min);",
                     "const double stat = p->up - p->up_min;"),
    "ph_alarm_inclusive": ("if (stat > o->ph_lambda) {", "if (stat >= o->ph_lambda) {"),
    "ph_downward_sign": ("p->dn += (rbar - r) - o->ph_delta;", "p->dn += (r - rbar) - o->ph_delta;"),
    "ph_window_off_by_one": ("t - o->ph_last[i] >= o->ph_window", "t - o->ph_last[i] > o->ph_window"),
    "ph_min_rounds_ignored": ("t >= o->ph_min_rounds && ", ""),
    "greedy_scores_with_bonus": ("U[k] = greedy ? m : m + alpha * w;", "U[k] = m + alpha * w;"),
    "coarse_grid_from_bottom": ("return k >= lo && k <= hi && (hi - k) % st == 0;",
                                "return k >= lo && k <= hi && (k - lo) % st == 0;"),
    "nonsticky_ignores_action_space": ("                act0[k] = in_space(o, i, k);\n", "                act0[k] = 1;\n"),
    "nonsticky_removals_stay": ("                kp[k] = 1;\n", "                kp[k] = glob[k];\n"),
    "nonsticky_while_exploiting": ("if (prune_now && !o->sticky && !greedy)", "if (prune_now && !o->sticky)"),
    "nonsticky_never": ("if (prune_now && !o->sticky && !greedy)", "if (0)"),
    "refine_min_samples_off_by_one": ("n[k] >= o->refine_min_n", "n[k] > o->refine_min_n"),
    "refine_anchor_worst_mean": ("rs[k] / n[k] > rs[anchor] / n[anchor]",
                                 "rs[k] / n[k] < rs[anchor] / n[anchor]"),
    "refine_predictive_from_maturity_plus_one": ("if (t < o->refine_mature) {", "if (t <= o->refine_mature) {"),
    "refine_window_one_sided": ("o->win[3 * i] = anchor - o->refine_half > 0 ? anchor - o->refine_half : 0;",
                                "o->win[3 * i] = anchor;"),
    "refine_keeps_coarse_stride": ("    o->win[3 * i + 2] = 1;\n}", "    o->win[3 * i + 2] = o->refine_stride;\n}"),
    "refine_period_off_by_one": ("(t % o->refine_period) == 0", "((t + 1) % o->refine_period) == 0"),
    "refine_candidates_include_pruned": ("if (glob[k] && in_space(o, i, k) && n[k] >= o->refine_min_n &&",
                                         "if (in_space(o, i, k) && n[k] >= o->refine_min_n &&"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(_SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not found exactly once"
    mutant_src = tmp_path / "mutant.c"
    mutant_src.write_text(src.replace(old, new))
    lib_path = build_library(str(mutant_src), str(tmp_path / "libmutant.so"))
    lib = load_library(lib_path)
    caught = []
    for pin in pins.ALL_PINS:
        try:
            pin(lib)
        except AssertionError:
            caught.append(pin.__name__)
        except (ValueError, FloatingPointError, ZeroDivisionError, IndexError):
            caught.append(pin.__name__)
    assert caught, f"mutant {name} survived every pin"


def test_unmutated_copy_passes(tmp_path):
    lib_path = build_library(_SRC, str(tmp_path / "libcopy.so"))
    lib = load_library(lib_path)
    for pin in pins.ALL_PINS:
        pin(lib)
