"""The parity harness itself, on the CPU: a record made by the oracle passes
the open-loop comparison, and a record with one planted difference fails it.
(The record here is the oracle's own, so these tests say nothing about the
GPU; they check that the comparison would catch what it is meant to.)"""
import numpy as np
import pytest

import parity
from oracle import Oracle

FAST_PH = dict(ph_delta=0.05, ph_lambda=5.0, ph_window=40, ph_min_rounds=60)


def _inputs(seed, T, B, d):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((T, B, d))
    X[:, :, 0] = 1.0
    R = rng.uniform(-2.0, 0.0, size=(T, B))
    R[T // 2:, ::2] -= 1.5
    return X.astype(np.float32).astype(np.float64), R.astype(np.float32).astype(np.float64)


def _record(cfg, X, R):
    """Run the oracle and keep what the GPU run records, in the GPU's formats."""
    T, B, _ = X.shape
    K = cfg["K"]
    ora = Oracle(B, K, cfg["d"], cfg["lam"], cfg["alpha0"], cfg["sched"], cfg["prune"], cfg["period"])
    if cfg.get("exploit"):
        ora.set_exploit(True, **cfg["exploit"])
    if cfg.get("refine"):
        ora.set_refine(True, **cfg["refine"])
    win = np.empty((T, B, 3), np.int32)
    KW = (K + 31) // 32
    acts = np.empty((T, B), np.int32)
    masks = np.zeros((T, B, KW), np.int64)
    scores = np.empty((T, B, 2, K))
    ph = np.empty((T, B, 9), np.int32)
    r_prev = None
    for t in range(T):
        ucb, lcb, keep, action = ora.decide(X[t], r_prev)
        ora.commit(X[t], action, keep)
        win[t] = [ora.window(i) for i in range(B)]
        acts[t] = action
        for k in range(K):
            masks[t, :, k // 32] |= keep[:, k].astype(np.int64) << (k % 32)
        scores[t, :, 0], scores[t, :, 1] = ucb, lcb
        for i in range(B):
            st, margin, last, mode = ora.page_hinkley(i)
            ph[t, i, 0] = mode
            ph[t, i, 1:7] = st.astype(np.float32).view(np.int32)
            ph[t, i, 7] = last
            ph[t, i, 8] = np.float32(margin).view(np.int32)
        r_prev = R[t]
    return acts, masks.astype(np.uint32).view(np.int32), scores.astype(np.float32).astype(np.float64), ph, win


CFG = dict(B=6, K=12, d=8, lam=1.0, alpha0=0.5, sched=0, prune=1, period=20, exploit=FAST_PH)


def test_oracle_record_passes():
    X, R = _inputs(3, 150, CFG["B"], CFG["d"])
    a, m, s, ph, _ = _record(CFG, X, R)
    assert (ph[-1, :, 0] >= 0).any() and (ph[:, :, 7] > 0).any()
    st = parity.compare_open_loop("self", CFG, X, R, a, m, s, g_ph=ph)
    assert st["greedy_decisions"] > 0 and st["forced_ph"] == 0


@pytest.mark.parametrize("plant", ["switch_round", "alarm_round", "statistic", "greedy_score"])
def test_planted_difference_fails(plant):
    X, R = _inputs(3, 150, CFG["B"], CFG["d"])
    a, m, s, ph, _ = _record(CFG, X, R)
    modes = ph[-1, :, 0]
    i = int(np.flatnonzero(modes >= 0)[0])
    t_sw = int(modes[i])
    if plant == "switch_round":         # the record switches one step late
        ph[t_sw, i, 0] = -1
    elif plant == "alarm_round":        # an alarm one round off
        t = int(np.flatnonzero(ph[:, :, 7].max(axis=1) > 0)[0])
        j = int(np.flatnonzero(ph[t, :, 7] > 0)[0])
        ph[t:, j, 7] += 1
    elif plant == "statistic":          # the running mean off by 1e-3
        st = ph[t_sw // 2, i, 1:7].view(np.float32)
        st[1] += np.float32(1e-3)
    else:                               # a greedy score off by 1e-3
        s[t_sw + 1, i, :, int(a[t_sw + 1, i])] += 1e-3
    with pytest.raises(parity.ParityError):
        parity.compare_open_loop("planted", CFG, X, R, a, m, s, g_ph=ph)


RCFG = dict(B=4, K=30, d=4, lam=1.0, alpha0=0.5, sched=0, prune=1, period=13,
            refine=dict(refine_period=6, refine_stride=5, refine_half=3, refine_mature=24,
                        refine_min_n=2))


def test_oracle_record_with_refinement_passes():
    X, R = _inputs(8, 60, RCFG["B"], RCFG["d"])
    a, m, s, _, win = _record(RCFG, X, R)
    assert (win[:, :, 2] == 1).any()
    st = parity.compare_open_loop("self-refine", RCFG, X, R, a, m, s, g_win=win)
    assert st["refinements"] > 0 and st["forced_window"] == 0


@pytest.mark.parametrize("plant", ["predictive_shift", "statistical_far_anchor", "stride"])
def test_planted_window_difference_fails(plant):
    X, R = _inputs(8, 60, RCFG["B"], RCFG["d"])
    a, m, s, _, win = _record(RCFG, X, R)
    if plant == "predictive_shift":            # one arm off after a predictive refinement
        t = 30
        win[t:, 0, :2] = np.minimum(win[t:, 0, :2] + 1, RCFG["K"] - 1)
    elif plant == "statistical_far_anchor":    # a window around the arm with the worst mean
        t = 6
        win[t:, 1] = (0, 6, 1)
    else:                                      # the coarse grid kept after a refinement
        t = 12
        win[t:, 2, 2] = RCFG["refine"]["refine_stride"]
    with pytest.raises(parity.ParityError):
        parity.compare_open_loop("planted-window", RCFG, X, R, a, m, s, g_win=win)


# ---- the vectorised every-instance comparison (closed loop, no scores) ----

def _closed_record(wl):
    """The oracle's own closed-loop run, kept in the GPU run's formats."""
    from agft_workloads import exogenous
    from oracle import run_closed_loop
    arrivals, noise = exogenous(wl, None, wl.T)
    out = run_closed_loop(wl, arrivals, noise, T=wl.T, record=True)
    T, n, K = out["keep"].shape
    words = np.zeros((T, n, (K + 31) // 32), np.int64)
    for k in range(K):
        words[:, :, k // 32] |= out["keep"][:, :, k].astype(np.int64) << (k % 32)
    rec = dict(a=out["actions"].copy(), mask=words.astype(np.uint32).view(np.int32),
               x=out["x"].astype(np.float32), r=out["r"].astype(np.float32))
    return rec, out


def _wl():
    from agft_workloads import get_workload
    return get_workload(3, B=6, K=24, T=120)


def test_every_instance_oracle_record_passes():
    wl = _wl()
    rec, out = _closed_record(wl)
    assert not out["keep"][-1].all()   # pruning happened
    st = parity.compare_every_instance(wl, wl.T, rec, range(wl.B))
    assert st["decisions"] == wl.B * wl.T and st["forced"] == 0 and st["forced_prune"] == 0
    assert st["exact_tie_steps"] > 0   # untouched arms at the start
    # any subset of the batch, in order
    sub = [1, 4]
    st = parity.compare_every_instance(wl, wl.T, {k: v[:, sub] for k, v in rec.items()}, sub)
    assert st["decisions"] == 2 * wl.T


@pytest.mark.parametrize("plant", ["action", "context", "reward", "prune", "exact_tie"])
def test_every_instance_planted_difference_fails(plant):
    wl = _wl()
    rec, out = _closed_record(wl)
    ucb, keep = out["ucb"], out["keep"]
    if plant == "action":
        # the second-best arm where the top two are far apart
        u = np.where(keep, ucb, -np.inf)
        top = np.sort(u, axis=2)
        gap = top[..., -1] - top[..., -2]
        t, i = map(int, np.argwhere(gap[60:] > 1e-2)[0])
        t += 60
        rec["a"][t, i] = int(np.argsort(u[t, i])[-2])
    elif plant == "context":
        rec["x"][70, 2, 3] += 1e-3
    elif plant == "reward":
        rec["r"][70, 3] += 1e-3
    elif plant == "prune":
        # an arm far above the threshold dropped at the prune step
        t = wl.period
        i = 0
        lstar = np.where(np.isfinite(ucb[t, i]), out["lcb"][t, i], -np.inf).max()
        k = int(np.flatnonzero(keep[t, i] & (ucb[t, i] - lstar > 1e-2))[0])
        if k == int(rec["a"][t, i]):
            k = int(np.flatnonzero(keep[t, i] & (ucb[t, i] - lstar > 1e-2))[1])
        words = rec["mask"].view(np.uint32)
        words[t:, i, k // 32] &= np.uint32(0xFFFFFFFF ^ (1 << (k % 32)))
    else:
        # step 0: every arm untouched and bit-identical; the lowest index must win
        assert (ucb[0, 0] == ucb[0, 0, 0]).all()
        rec["a"][0, 0] = 1
    expect = {"action": "action mismatch", "context": "context mismatch", "reward": "reward mismatch",
              "prune": "prune mismatch", "exact_tie": "exact tie"}[plant]
    with pytest.raises(parity.ParityError, match=expect):
        parity.compare_every_instance(wl, wl.T, rec, range(wl.B))


def test_every_instance_with_paper_rules_passes():
    from agft_workloads import get_workload
    wl = get_workload("cfg2p", B=6, T=200)
    rec, out = _closed_record(wl)
    assert wl.prune & 14 and not out["keep"][-1].all()
    st = parity.compare_every_instance(wl, wl.T, rec, range(wl.B))
    assert st["decisions"] == wl.B * wl.T and st["forced"] == 0 and st["forced_rules"] == 0


def test_every_instance_rule_removal_planted_fails():
    """An arm that the paper's rules removed far from any threshold, kept in
    the record's mask from then on."""
    from agft_workloads import get_workload
    wl = get_workload("cfg2p", B=6, T=200)
    rec, out = _closed_record(wl)
    keep = out["keep"]
    gone = keep[:-1] & ~keep[1:]                 # removed at step t + 1
    t, i, k = map(int, np.argwhere(gone)[0])
    t += 1
    words = rec["mask"].view(np.uint32)
    words[t:, i, k // 32] |= np.uint32(1 << (k % 32))
    with pytest.raises(parity.ParityError, match="prune mismatch"):
        parity.compare_every_instance(wl, wl.T, rec, range(wl.B))


def _closed_record_full(wl):
    """As _closed_record, with the test words and action spaces after each step."""
    from agft_workloads import exogenous
    from oracle import run_closed_loop
    arrivals, noise = exogenous(wl, None, wl.T)
    T, B = wl.T, wl.B
    ph = np.empty((T, B, 9), np.int32)
    win = np.empty((T, B, 3), np.int32)
    box = {}

    def commit(t):
        o = box["ora"]
        if wl.exploit:
            stats, margin, last, mode = o.page_hinkley_all()
            ph[t, :, 0] = mode
            ph[t, :, 1:7] = stats.astype(np.float32).view(np.int32)
            ph[t, :, 7] = last
            ph[t, :, 8] = margin.astype(np.float32).view(np.int32)
        win[t] = o.windows()
    out = run_closed_loop(wl, arrivals, noise, T=T, record=True,
                          on_create=lambda o: box.__setitem__("ora", o), on_commit=commit)
    K = wl.K
    words = np.zeros((T, B, (K + 31) // 32), np.int64)
    for k in range(K):
        words[:, :, k // 32] |= out["keep"][:, :, k].astype(np.int64) << (k % 32)
    rec = dict(a=out["actions"].copy(), mask=words.astype(np.uint32).view(np.int32),
               x=out["x"].astype(np.float32), r=out["r"].astype(np.float32), ph=ph, win=win)
    return rec, out


def test_every_instance_switch_and_refinement_pass():
    from agft_workloads import get_workload
    wl = get_workload("cfg2e", B=6, T=300)
    rec, _ = _closed_record_full(wl)
    assert (rec["ph"][-1, :, 0] >= 0).any()
    st = parity.compare_every_instance(wl, wl.T, rec, range(wl.B))
    assert st["greedy_decisions"] > 0 and st["forced_ph"] == 0 and st["forced"] == 0
    wl = get_workload("cfg2r", B=6, T=220)
    rec, _ = _closed_record_full(wl)
    st = parity.compare_every_instance(wl, wl.T, rec, range(wl.B))
    assert st["refinements"] > 0 and st["forced_window"] == 0 and st["forced"] == 0


@pytest.mark.parametrize("plant", ["switch_late", "statistic", "window"])
def test_every_instance_switch_or_window_planted_fails(plant):
    from agft_workloads import get_workload
    if plant == "window":
        wl = get_workload("cfg2r", B=6, T=220)
        rec, _ = _closed_record_full(wl)
        t = 150                                  # after a refinement: a window one arm off
        rec["win"][t:, 2, :2] += 1
        expect = "action space differs"
    else:
        wl = get_workload("cfg2e", B=6, T=300)
        rec, _ = _closed_record_full(wl)
        modes = rec["ph"][-1, :, 0]
        i = int(np.flatnonzero(modes >= 0)[0])
        t_sw = int(modes[i])
        if plant == "switch_late":
            rec["ph"][t_sw, i, 0] = -1
            expect = "Page-Hinkley test differs"
        else:                                    # the running mean off by 1e-3
            st = rec["ph"][t_sw // 2, i, 1:7].view(np.float32)
            st[1] += np.float32(1e-3)
            expect = "Page-Hinkley statistics differ"
    with pytest.raises(parity.ParityError, match=expect):
        parity.compare_every_instance(wl, wl.T, rec, range(wl.B))
