"""Closed-loop driver of the oracle: environment + bandit, in fp64.

Test infrastructure only.
"""
import numpy as np

from .env import Env
from .oracle import Oracle


def run_closed_loop(wl, arrivals, noise, T=None, on_decide=None, record=False, lib=None,
                    margins=False, on_create=None, on_commit=None):
    """Run T decisions of len(instances) tuners against the fp64 environment.

    arrivals, noise: [T+1][n] exogenous draws (agft_workloads.exogenous).
    on_decide(t, x, r_prev, ucb, lcb, keep, action[, margins]) may return
    (action, keep) to commit instead of the oracle's own decision (a
    near-tied alternative); with margins=True it also receives the distances
    of the pruning-rule comparisons from their thresholds.
    Returns a dict with the oracle object, actions [T][n] and, if record is
    set, contexts [T][n][d], rewards [T][n] (reward of decision t) and
    ucb/lcb [T][n][K].  on_create(oracle) is called once the oracle exists,
    on_commit(t) after each decision is committed.
    """
    T = wl.T if T is None else int(T)
    env = Env(wl, arrivals, noise, T)
    n = env.n
    ora = Oracle.from_workload(wl, B=n, lib=lib)
    if on_create is not None:
        on_create(ora)
    x = env.reset()
    r_prev = None
    actions = np.empty((T, n), dtype=np.int32)
    rec = dict(x=[], r=[], ucb=[], lcb=[], keep=[]) if record else None
    for t in range(T):
        if margins:
            ucb, lcb, keep, action, marg = ora.decide(x, r_prev, margins=True)
        else:
            ucb, lcb, keep, action = ora.decide(x, r_prev)
        if on_decide is not None:
            args = (t, x, r_prev, ucb, lcb, keep, action) + ((marg,) if margins else ())
            over = on_decide(*args)
            if over is not None:
                action, keep = over
        ora.commit(x, action, keep)
        if on_commit is not None:
            on_commit(t)
        actions[t] = action
        if record:
            rec["x"].append(x.copy()); rec["ucb"].append(ucb); rec["lcb"].append(lcb)
            rec["keep"].append(keep)
        r_prev, x = env.step(t, action)
        if record:
            rec["r"].append(r_prev.copy())
    ora.flush(r_prev)
    out = dict(oracle=ora, actions=actions, env=env)
    if record:
        for key in rec:
            out[key] = np.stack(rec[key])
    return out
