"""Comparison of recorded GPU runs with the fp64 oracle.

The oracle makes its own decisions.  Only where the paper's method admits
several answers does it take the GPU's: an arm whose UCB is within TIE of the
best (the argmax is not unique at the precision the scores carry) and a prune
decision whose UCB is within TIE of the threshold.  Exact ties in the oracle
(arms with bit-identical scores, e.g. untouched arms) are not ambiguous: the
lowest index must win on both sides.

Closed loop (compare): the oracle also runs its own fp64 environment on the
same exogenous draws, so GPU contexts and rewards are checked too.
Open loop (compare_open_loop): both sides get the same given contexts and
rewards.

The Page-Hinkley test behind the switch to exploitation runs in double
precision in the oracle and in single precision on the GPU, so its running
sums are compared within PH_TOL, and an alarm that one side raised and the
other did not is accepted only where the oracle's margin (lambda minus the
larger statistic) was within PH_TIE of zero, relative to the magnitude of the
running sums whose difference the statistic is; the oracle then adopts the
GPU's test state (and, for that step, the GPU's decision, since the two
scored in different modes).  Alarm rounds and the switch round are integers:
away from such near-threshold alarms they must be identical.

The refinement of the action space is compared after every committed step:
the windows must be identical, except at a statistical refinement whose two
candidate anchors have mean rewards within MEAN_TIE of each other (fp32 sums
on the GPU, fp64 in the oracle); the oracle then adopts the GPU's window.
"""
import numpy as np

from agft_workloads import exogenous
from oracle import Oracle, run_closed_loop

SCORE_TOL = 1e-4   # |s_gpu - s_oracle| <= SCORE_TOL * max(1, |s_oracle|): relative for |s| >= 1,
                   # absolute below (rewards and scores are O(1), many below 1 in magnitude)
TIE = 1e-5         # score gaps at or below this (times max(1, |score|)) are near-ties
ENV_TOL = 1e-5     # contexts and rewards: fp32 environment vs fp64 environment
PH_TOL = 1e-4      # Page-Hinkley running sums: |s_gpu - s_oracle| <= PH_TOL * max(1, |s_oracle|)
PH_TIE = 1e-4      # |lambda - statistic| <= PH_TIE * max(1, |running sums|): the alarm could go either way
MEAN_TIE = 1e-4    # mean rewards this close (relative): either can anchor a refinement


def ph_tie_scale(*stats):
    """Magnitude the Page-Hinkley statistic's rounding scales with: the
    largest running sum (m+, min m+, m-, min m-) of either side, at least 1
    (one side has just restarted after an alarm, the other has not)."""
    return max([1.0] + [float(np.max(np.abs(np.asarray(s, dtype=np.float64)[2:6]))) for s in stats])


def mask_words_to_bool(words, K):
    words = np.asarray(words).astype(np.int64) & 0xFFFFFFFF
    k = np.arange(K)
    return ((words[..., k // 32] >> (k % 32)) & 1).astype(bool)


class ParityError(AssertionError):
    pass


class Checker:
    def __init__(self, name, K, ids, g_a, g_keep, g_s=None, g_x=None, g_r=None, rules=0,
                 cascade_k=0, g_ph=None, g_win=None, refine=None, g_gap=None):
        self.name, self.K, self.ids = name, K, list(ids)
        # g_gap [T][n]: top-two gap of each decision (largest kept score minus
        # the second), checked against the oracle's within both scores' tolerance
        self.g_gap = g_gap
        self.g_a, self.g_keep, self.g_s, self.g_x, self.g_r = g_a, g_keep, g_s, g_x, g_r
        self.rules, self.cascade_k = rules, cascade_k
        # g_ph [T][n][9] int32: mode, Page-Hinkley n, mean, m+, min m+, m-, min m-,
        # last alarm round, last margin (fp32 bits), after each step
        self.g_ph = g_ph
        # g_win [T][n][3] int32: action space lo, hi, stride after each step;
        # refine: the refinement parameters (period, half, mature, min_n)
        self.g_win, self.refine = g_win, refine
        self.oracle = None
        self.st = dict(max_score_err=0.0, max_ctx_err=0.0, max_reward_err=0.0, forced=0,
                       forced_prune=0, forced_rules=0, exact_tie_steps=0, decisions=0,
                       no_decision=0, max_ph_err=0.0, forced_ph=0, forced_mode=0,
                       greedy_decisions=0, refinements=0, forced_window=0, max_gap_err=0.0,
                       max_rel_err_abs_ge_1=0.0, max_abs_err_abs_lt_1=0.0)

    def _anchor(self, lo, hi):
        h = self.refine["refine_half"]
        if lo > 0:
            return lo + h
        if hi < self.K - 1:
            return hi - h
        return None

    def after_commit(self, t):
        """Compare the action spaces once step t is committed."""
        if self.g_win is None:
            return
        rf = self.refine
        for i in range(len(self.ids)):
            o_win = tuple(self.oracle.window(i))
            g_win = tuple(int(v) for v in self.g_win[t, i])
            if t > 0 and t % rf["refine_period"] == 0 and g_win[2] == 1:
                self.st["refinements"] += 1
            if o_win == g_win:
                continue
            stat_step = t > 0 and t % rf["refine_period"] == 0 and t < rf["refine_mature"]
            a_o, a_g = self._anchor(*o_win[:2]), self._anchor(*g_win[:2])
            ok = stat_step and a_o is not None and a_g is not None and g_win[2] == 1
            if ok:
                st = self.oracle.get(i)
                n, rs = st["nsel"], st["rsum"]
                ok = n[a_g] >= rf["refine_min_n"] and n[a_o] >= rf["refine_min_n"]
                if ok:
                    m_o, m_g = rs[a_o] / n[a_o], rs[a_g] / n[a_g]
                    ok = abs(m_o - m_g) <= MEAN_TIE * max(1.0, abs(m_o))
            if not ok:
                self.fail(f"action space differs after t={t}, instance {self.ids[i]}: GPU {g_win}, "
                          f"oracle {o_win}")
            self.oracle.set_window(i, *g_win)
            self.st["forced_window"] += 1

    def bind(self, oracle):
        """The oracle whose Page-Hinkley state is checked (and forced)."""
        self.oracle = oracle

    def _check_ph(self, t, i):
        """Compare instance i's test state after step t; returns True when the
        two sides scored this step in different modes (decision forced)."""
        g = np.asarray(self.g_ph[t, i], dtype=np.int32)
        g_mode, g_last = int(g[0]), int(g[7])
        g_stats = g[1:7].view(np.float32).astype(np.float64)
        g_margin = float(g[8:9].view(np.float32)[0])
        o_stats, o_margin, o_last, o_mode = self.oracle.page_hinkley(i)
        if g_mode == o_mode and g_last == o_last:
            err = np.abs(g_stats - o_stats) / np.maximum(1.0, np.abs(o_stats))
            self.st["max_ph_err"] = max(self.st["max_ph_err"], float(err.max()))
            if err.max() > PH_TOL:
                self.fail(f"Page-Hinkley statistics differ at t={t}, instance {self.ids[i]}: "
                          f"{g_stats} vs {o_stats}")
            return False
        if g_last == o_last or abs(o_margin) > PH_TIE * ph_tie_scale(g_stats, o_stats):
            self.fail(f"Page-Hinkley test differs at t={t}, instance {self.ids[i]}: GPU mode {g_mode}, "
                      f"last alarm {g_last}; oracle mode {o_mode}, last alarm {o_last}, "
                      f"margin {o_margin}")
        self.oracle.set_page_hinkley(i, g_stats, g_margin, g_last, g_mode)
        self.st["forced_ph"] += 1
        if (g_mode >= 0) != (o_mode >= 0):
            self.st["forced_mode"] += 1
            return True
        return False

    def fail(self, msg):
        raise ParityError(f"{self.name}: {msg}")

    def _rules_ambiguous(self, margins, k):
        """Arm k's removal by the paper's rules (bits 2, 4, 8) could go either
        way: its own comparison, or that of a higher arm whose cascade covers
        it, sits within TIE of the threshold."""
        if margins is None:
            return False
        if margins[k] <= TIE:
            return True
        if self.rules & 8:
            hi = np.arange(self.K)
            return bool(np.any((hi > k) & (hi < self.cascade_k) & (margins <= TIE)))
        return False

    def __call__(self, t, x, r_prev, ucb, lcb, keep, action, margins=None):
        st, ids = self.st, self.ids
        if self.g_x is not None:
            ex = np.abs(self.g_x[t] - x) / np.maximum(1.0, np.abs(x))
            ex = np.where(np.isfinite(x), ex, 0.0)
            st["max_ctx_err"] = max(st["max_ctx_err"], float(ex.max()))
            if ex.max() > ENV_TOL:
                i = int(np.argmax(ex.max(axis=1)))
                self.fail(f"context mismatch at t={t}, instance {ids[i]}: {self.g_x[t, i]} vs {x[i]}")
        if self.g_r is not None and t > 0:
            er = np.abs(self.g_r[t - 1] - r_prev) / np.maximum(1.0, np.abs(r_prev))
            st["max_reward_err"] = max(st["max_reward_err"], float(er.max()))
            if er.max() > ENV_TOL:
                self.fail(f"reward mismatch at t={t - 1}: max rel err {er.max():.3e}")
        act = np.isfinite(ucb)
        commit_keep = keep.copy()
        commit_a = action.copy()
        for i in range(len(ids)):
            ga = int(self.g_a[t, i])
            if self.g_ph is not None:
                if self._check_ph(t, i):
                    commit_keep[i] = self.g_keep[t, i]
                    commit_a[i] = ga
                    continue
                if self.g_ph[t, i, 0] >= 0 and action[i] >= 0:
                    st["greedy_decisions"] += 1
            if self.g_s is not None:
                g_act = np.isfinite(self.g_s[t, i, 0])
                if not np.array_equal(g_act, act[i]):
                    diff = np.flatnonzero(g_act != act[i])
                    if not all(self._rules_ambiguous(None if margins is None else margins[i], k)
                               for k in diff):
                        self.fail(f"active sets differ at t={t}, instance {ids[i]}, arms {diff}")
                    # a near-threshold pruning rule decided differently: take the GPU's set
                    st["forced_rules"] += 1
                    commit_keep[i] = self.g_keep[t, i]
                    commit_a[i] = ga
                    continue
                for row, ref in ((0, ucb[i]), (1, lcb[i])):
                    with np.errstate(invalid="ignore"):
                        err = np.where(act[i], np.abs(self.g_s[t, i, row] - ref) / np.maximum(1.0, np.abs(ref)),
                                       0.0)
                    st["max_score_err"] = max(st["max_score_err"], float(err.max()))
                    # the same errors split by magnitude: relative where |s| >= 1,
                    # absolute below (where the bar's floor of 1 makes it absolute)
                    big = act[i] & (np.abs(ref) >= 1.0)
                    if big.any():
                        st["max_rel_err_abs_ge_1"] = max(st["max_rel_err_abs_ge_1"], float(err[big].max()))
                    small = act[i] & ~big
                    if small.any():
                        st["max_abs_err_abs_lt_1"] = max(st["max_abs_err_abs_lt_1"], float(err[small].max()))
                    if err.max() > SCORE_TOL:
                        k = int(np.argmax(err))
                        self.fail(f"score mismatch at t={t}, instance {ids[i]}, arm {k}: "
                                  f"{self.g_s[t, i, row, k]!r} vs {ref[k]!r}")
            if action[i] < 0:
                st["no_decision"] += 1
                if ga != -1:
                    self.fail(f"GPU decided on a non-finite context at t={t}, instance {ids[i]}")
                continue
            if not np.array_equal(self.g_keep[t, i], keep[i]):
                lstar = lcb[i][act[i]].max()
                diff = np.flatnonzero(self.g_keep[t, i] != keep[i])
                amb = np.abs(ucb[i, diff] - lstar) <= TIE * max(1.0, abs(lstar))
                if not amb.all():
                    self.fail(f"prune mismatch at t={t}, instance {ids[i]}, arms {diff[~amb]}")
                st["forced_prune"] += 1
                commit_keep[i] = self.g_keep[t, i]
            kp = commit_keep[i]
            u = np.where(kp, ucb[i], -np.inf)
            ustar = u.max()
            own = int(np.flatnonzero(u == ustar)[0])
            near = np.flatnonzero(kp & (ustar - ucb[i] <= TIE * max(1.0, abs(ustar))))
            st["decisions"] += 1
            if ga not in near:
                gu = ucb[i, ga] if 0 <= ga < self.K else None
                self.fail(f"action mismatch at t={t}, instance {ids[i]}: GPU {ga} (UCB {gu}), "
                          f"oracle {own} (UCB {ustar})")
            if len(near) > 1 and np.all(ucb[i, near] == ustar):
                st["exact_tie_steps"] += 1
                if ga != own:
                    self.fail(f"exact tie broken wrongly at t={t}, instance {ids[i]}: {ga} vs {own}")
            if self.g_gap is not None:
                top = np.sort(u[np.isfinite(u)])[::-1]
                o_gap = top[0] - top[1] if top.size > 1 else np.inf
                g_gap = float(self.g_gap[t, i])
                if np.isinf(o_gap):
                    ok = np.isinf(g_gap) and g_gap > 0
                    err = 0.0
                else:
                    err = abs(g_gap - o_gap) / max(1.0, abs(ustar))
                    ok = err <= 2 * SCORE_TOL
                st["max_gap_err"] = max(st["max_gap_err"], err)
                if not ok:
                    self.fail(f"top-two gap differs at t={t}, instance {ids[i]}: GPU {g_gap}, oracle {o_gap}")
            if ga != own:
                st["forced"] += 1
            commit_a[i] = ga
        return commit_a, commit_keep

    def finish(self):
        self.st["forced_rate"] = self.st["forced"] / max(1, self.st["decisions"])
        return self.st


class EveryInstanceChecker:
    """The comparison of Checker for runs recorded without scores, vectorised
    over instances so that it covers every instance of a full-size batch:
    contexts, rewards, prune decisions and actions at every step, under the
    same near-tie rules (where the oracle's fp64 scores leave the choice
    open, it adopts the GPU's).  With the paper's rules (bits 2, 4, 8) an
    arm may also be kept or removed differently when its rule comparison, or
    that of a higher arm whose cascade covers it, sat within TIE of the
    threshold; the oracle then adopts the GPU's active set and action.  With
    the switch, the test state after every step (within PH_TOL; an alarm one
    side raised alone only where the oracle's margin was within PH_TIE, then
    adopted with the GPU's decision); with the refinement, the action space
    after every step (a different anchor only at a statistical refinement
    whose candidates' mean rewards were within MEAN_TIE, then adopted): the
    rules of Checker, on every instance at once.

    g_a [T][n] actions, g_words [T][n][KW] mask words after each step,
    g_x [T][n][d] contexts, g_r [T][n] rewards (reward of decision t),
    g_ph [T][n][9] test words and g_win [T][n][3] action spaces after each
    step (with the switch and the refinement)."""

    def __init__(self, name, K, ids, g_a, g_words, g_x, g_r, rules=0, cascade_k=0, g_ph=None,
                 g_win=None, refine=None):
        self.name, self.K, self.ids = name, K, np.asarray(ids)
        self.g_a, self.g_words, self.g_x, self.g_r = g_a, g_words, g_x, g_r
        self.rules, self.cascade_k = rules, cascade_k
        self.g_ph, self.g_win, self.refine = g_ph, g_win, refine
        self.oracle = None
        self.st = dict(max_ctx_err=0.0, max_reward_err=0.0, forced=0, forced_prune=0, forced_rules=0,
                       exact_tie_steps=0, decisions=0, no_decision=0, instances=len(self.ids),
                       max_ph_err=0.0, forced_ph=0, forced_mode=0, greedy_decisions=0,
                       refinements=0, forced_window=0)

    def bind(self, oracle):
        self.oracle = oracle

    def _check_ph(self, t):
        """Test state of every instance after step t; returns the rows whose
        decision the two sides took in different modes (adopted as the GPU's)."""
        g = np.asarray(self.g_ph[t], dtype=np.int32)
        g_mode, g_last = g[:, 0].astype(np.int64), g[:, 7].astype(np.int64)
        g_stats = np.ascontiguousarray(g[:, 1:7]).view(np.float32).astype(np.float64)
        g_margin = np.ascontiguousarray(g[:, 8]).view(np.float32).astype(np.float64)
        o_stats, o_margin, o_last, o_mode = self.oracle.page_hinkley_all()
        same = (g_mode == o_mode) & (g_last == o_last)
        if same.any():
            a, b = g_stats[same], o_stats[same]
            err = np.abs(a - b) / np.maximum(1.0, np.abs(b))
            self.st["max_ph_err"] = max(self.st["max_ph_err"], float(err.max()))
            if err.max() > PH_TOL:
                i = int(np.flatnonzero(same)[np.argmax(err.max(axis=1))])
                self.fail(f"Page-Hinkley statistics differ at t={t}, instance {self.ids[i]}: "
                          f"{g_stats[i]} vs {o_stats[i]}")
        mode_rows = np.zeros(len(g_mode), dtype=bool)
        for i in np.flatnonzero(~same):
            tie = PH_TIE * ph_tie_scale(g_stats[i], o_stats[i])
            if g_last[i] == o_last[i] or abs(float(o_margin[i])) > tie:
                self.fail(f"Page-Hinkley test differs at t={t}, instance {self.ids[i]}: GPU mode "
                          f"{g_mode[i]}, last alarm {g_last[i]}; oracle mode {o_mode[i]}, last alarm "
                          f"{o_last[i]}, margin {o_margin[i]}")
            self.oracle.set_page_hinkley(int(i), g_stats[i], float(g_margin[i]), int(g_last[i]), int(g_mode[i]))
            self.st["forced_ph"] += 1
            if (g_mode[i] >= 0) != (o_mode[i] >= 0):
                self.st["forced_mode"] += 1
                mode_rows[i] = True
        return mode_rows, g_mode

    def after_commit(self, t):
        """Action spaces of every instance once step t is committed."""
        if self.g_win is None:
            return
        rf = self.refine
        g = np.asarray(self.g_win[t], dtype=np.int64)
        o = self.oracle.windows().astype(np.int64)
        if t > 0 and t % rf["refine_period"] == 0:
            self.st["refinements"] += int((g[:, 2] == 1).sum())
        stat_step = t > 0 and t % rf["refine_period"] == 0 and t < rf["refine_mature"]
        h = rf["refine_half"]

        def anchor(lo, hi):
            if lo > 0:
                return lo + h
            if hi < self.K - 1:
                return hi - h
            return None
        for i in np.flatnonzero((g != o).any(axis=1)):
            a_o, a_g = anchor(o[i, 0], o[i, 1]), anchor(g[i, 0], g[i, 1])
            ok = stat_step and a_o is not None and a_g is not None and g[i, 2] == 1
            if ok:
                st = self.oracle.get(int(i))
                n, rs = st["nsel"], st["rsum"]
                ok = n[a_g] >= rf["refine_min_n"] and n[a_o] >= rf["refine_min_n"]
                if ok:
                    m_o, m_g = rs[a_o] / n[a_o], rs[a_g] / n[a_g]
                    ok = abs(m_o - m_g) <= MEAN_TIE * max(1.0, abs(m_o))
            if not ok:
                self.fail(f"action space differs after t={t}, instance {self.ids[i]}: GPU "
                          f"{tuple(g[i])}, oracle {tuple(o[i])}")
            self.oracle.set_window(int(i), int(g[i, 0]), int(g[i, 1]), int(g[i, 2]))
            self.st["forced_window"] += 1

    def _rules_ambiguous(self, margins):
        """[n][K]: arm k's removal by rules 2/4/8 could go either way."""
        amb = margins <= TIE
        if self.rules & 8:
            arms = np.arange(self.K)
            cand = amb & (arms < self.cascade_k)
            top = np.where(cand.any(axis=1), self.K - 1 - np.argmax(cand[:, ::-1], axis=1), -1)
            amb = amb | (arms[None, :] < top[:, None])
        return amb

    def fail(self, msg):
        raise ParityError(f"{self.name}: {msg}")

    def __call__(self, t, x, r_prev, ucb, lcb, keep, action, margins=None):
        st, K = self.st, self.K
        gx = np.asarray(self.g_x[t], dtype=np.float64)
        with np.errstate(invalid="ignore"):
            ex = np.where(np.isfinite(x), np.abs(gx - x) / np.maximum(1.0, np.abs(x)), 0.0)
        st["max_ctx_err"] = max(st["max_ctx_err"], float(ex.max()))
        if ex.max() > ENV_TOL:
            i = int(np.argmax(ex.max(axis=1)))
            self.fail(f"context mismatch at t={t}, instance {self.ids[i]}: {gx[i]} vs {x[i]}")
        if t > 0:
            gr = np.asarray(self.g_r[t - 1], dtype=np.float64)
            er = np.abs(gr - r_prev) / np.maximum(1.0, np.abs(r_prev))
            st["max_reward_err"] = max(st["max_reward_err"], float(er.max()))
            if er.max() > ENV_TOL:
                i = int(np.argmax(er))
                self.fail(f"reward mismatch at t={t - 1}, instance {self.ids[i]}: {gr[i]} vs {r_prev[i]}")
        ga = np.asarray(self.g_a[t], dtype=np.int64)
        dec = action >= 0
        mode_rows = np.zeros(len(ga), dtype=bool)
        if self.g_ph is not None:
            mode_rows, g_mode = self._check_ph(t)
            self.st["greedy_decisions"] += int(((g_mode >= 0) & dec & ~mode_rows).sum())
        st["no_decision"] += int((~dec).sum())
        if np.any(~dec & (ga != -1)):
            i = int(np.flatnonzero(~dec & (ga != -1))[0])
            self.fail(f"GPU decided on a non-finite context at t={t}, instance {self.ids[i]}")
        act = np.isfinite(ucb)
        g_keep = mask_words_to_bool(self.g_words[t], K)
        commit_keep = keep.copy()
        diff = (g_keep != keep) & (dec & ~mode_rows)[:, None]
        rows = np.flatnonzero(diff.any(axis=1))
        by_rules = np.zeros(len(ga), dtype=bool)
        if rows.size:
            # a prune decision may differ only where the arm's UCB is within
            # TIE of the largest LCB over the active arms (rule 1), or where
            # the paper's rules could go either way
            lstar = np.where(act[rows], lcb[rows], -np.inf).max(axis=1)
            with np.errstate(invalid="ignore"):
                amb1 = np.abs(ucb[rows] - lstar[:, None]) <= TIE * np.maximum(1.0, np.abs(lstar))[:, None]
            amb_r = (self._rules_ambiguous(margins[rows]) if margins is not None
                     else np.zeros_like(amb1))
            bad = diff[rows] & ~(amb1 | amb_r)
            if bad.any():
                q = int(np.flatnonzero(bad.any(axis=1))[0])
                self.fail(f"prune mismatch at t={t}, instance {self.ids[rows[q]]}, "
                          f"arms {np.flatnonzero(bad[q])}")
            commit_keep[rows] = g_keep[rows]
            # where a rule decided differently the two sides scored different
            # sets: the GPU's decision is taken as it is
            by_rules[rows] = (diff[rows] & amb_r & ~amb1).any(axis=1)
            st["forced_rules"] += int(by_rules.sum())
            st["forced_prune"] += int(rows.size - by_rules.sum())
        u = np.where(commit_keep, ucb, -np.inf)
        ustar = u.max(axis=1)
        own = u.argmax(axis=1)          # the lowest index among exact maxima
        tol = TIE * np.maximum(1.0, np.abs(ustar))
        with np.errstate(invalid="ignore"):
            near = commit_keep & ((ustar[:, None] - ucb) <= tol[:, None])
        valid = (ga >= 0) & (ga < K)
        gac = np.clip(ga, 0, K - 1)
        skip = by_rules | mode_rows
        commit_keep[mode_rows] = g_keep[mode_rows]
        ok = ~dec | skip | (valid & near[np.arange(len(ga)), gac])
        if not ok.all():
            i = int(np.flatnonzero(~ok)[0])
            gu = ucb[i, ga[i]] if valid[i] else None
            self.fail(f"action mismatch at t={t}, instance {self.ids[i]}: GPU {ga[i]} (UCB {gu}), "
                      f"oracle {own[i]} (UCB {ustar[i]})")
        # exact ties (every near arm bit-identical to the best): lowest index on both sides
        exact = dec & ~skip & (near.sum(axis=1) > 1) & np.all(~near | (ucb == ustar[:, None]), axis=1)
        wrong = exact & (ga != own)
        if wrong.any():
            i = int(np.flatnonzero(wrong)[0])
            self.fail(f"exact tie broken wrongly at t={t}, instance {self.ids[i]}: {ga[i]} vs {own[i]}")
        st["exact_tie_steps"] += int(exact.sum())
        st["forced"] += int((dec & ~skip & (ga != own)).sum())
        st["decisions"] += int(dec.sum())
        return np.where(dec, ga, action).astype(np.int32), commit_keep

    def finish(self):
        self.st["forced_rate"] = self.st["forced"] / max(1, self.st["decisions"])
        return self.st


def compare_every_instance(wl, T, rec, ids):
    """Closed loop without scores: replay instances ids (any subset of the
    batch, in order) through the oracle and its environment and compare each
    one's contexts, rewards, prune decisions and actions at every step; raise
    ParityError on a violation.  rec: host arrays recorded for those
    instances, a [T][n], mask [T][n][KW], x [T][n][d], r [T][n], and ph
    [T][n][9] with the switch, win [T][n][3] with the refinement (the probe
    records of paper_2508_01744_amd.run_closed_loop)."""
    ids = np.asarray(ids)
    arrivals, noise = exogenous(wl, ids, T)
    chk = EveryInstanceChecker(wl.name, wl.K, ids, np.asarray(rec["a"]), np.asarray(rec["mask"]),
                               np.asarray(rec["x"]), np.asarray(rec["r"]), rules=wl.prune,
                               cascade_k=wl.cascade_k,
                               g_ph=np.asarray(rec["ph"]) if wl.exploit else None,
                               g_win=np.asarray(rec["win"]) if wl.refine else None,
                               refine=wl.refinement() if wl.refine else None)
    out = run_closed_loop(wl, arrivals, noise, T=T, on_decide=chk, margins=bool(wl.prune & 14),
                          on_create=chk.bind, on_commit=chk.after_commit)
    st = chk.finish()
    st["oracle"] = out["oracle"]
    return st


def compare(wl, T, probes, rec):
    """Closed loop: replay the probe instances through the oracle and its
    environment; raise ParityError on a violation.  rec: host tensors from
    paper_2508_01744_amd.run_closed_loop(probes=...)."""
    probes = list(probes)
    arrivals, noise = exogenous(wl, probes, T)
    chk = Checker(wl.name, wl.K, probes, rec["a"].numpy(),
                  mask_words_to_bool(rec["mask"].numpy(), wl.K),
                  rec["scores"].numpy().astype(np.float64) if "scores" in rec else None,
                  rec["x"].numpy().astype(np.float64), rec["r"].numpy().astype(np.float64),
                  rules=wl.prune, cascade_k=wl.cascade_k,
                  g_ph=rec["ph"].numpy() if wl.exploit else None,
                  g_win=rec["win"].numpy() if wl.refine else None,
                  refine=wl.refinement() if wl.refine else None,
                  g_gap=rec["gap"].numpy().astype(np.float64) if "gap" in rec else None)
    out = run_closed_loop(wl, arrivals, noise, T=T, on_decide=chk, margins=bool(wl.prune & 14),
                          on_create=chk.bind, on_commit=chk.after_commit)
    st = chk.finish()
    st["oracle"] = out["oracle"]
    return st


def compare_open_loop(name, cfg, X, R, g_a, g_masks, g_s, g_ph=None, g_win=None, g_gap=None):
    """Open loop: contexts X [T][B][d] and rewards R [T][B] (reward of the
    decision at t) given to both sides.  cfg: dict(B, K, d, lam, alpha0,
    sched, prune, period[, heuristics][, exploit][, refine]).  GPU records:
    actions [T][B], mask words [T][B][KW] after each step, scores
    [T][B][2][K], Page-Hinkley words [T][B][9] (when cfg has exploit), action
    spaces [T][B][3] (when cfg has refine)."""
    T = X.shape[0]
    ora = Oracle(cfg["B"], cfg["K"], cfg["d"], cfg["lam"], cfg["alpha0"], cfg["sched"],
                 cfg["prune"], cfg["period"])
    if not cfg.get("sticky", 1):
        ora.set_sticky(False)
    heur = cfg.get("heuristics")
    if heur:
        ora.set_heuristics(**heur)
    expl = cfg.get("exploit")
    if expl:
        ora.set_exploit(True, **expl)
    ref = cfg.get("refine")
    if ref:
        ora.set_refine(True, **ref)
    chk = Checker(name, cfg["K"], range(cfg["B"]), g_a, mask_words_to_bool(g_masks, cfg["K"]), g_s,
                  rules=cfg["prune"], cascade_k=(heur or {}).get("cascade_k", 0),
                  g_ph=g_ph if expl else None,
                  g_win=g_win if ref else None, refine=ref, g_gap=g_gap)
    chk.bind(ora)
    r_prev = None
    for t in range(T):
        ucb, lcb, keep, action, marg = ora.decide(X[t], r_prev, margins=True)
        a, k = chk(t, X[t], r_prev, ucb, lcb, keep, action, marg)
        ora.commit(X[t], a, k)
        chk.after_commit(t)
        r_prev = R[t]
    ora.flush(r_prev)
    st = chk.finish()
    st["oracle"] = ora
    return st
