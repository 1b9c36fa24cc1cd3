"""Checks that pin the fp64 oracle to the mathematics rather than to itself.

Each pin_* function takes an oracle library handle (oracle.load_library())
and raises AssertionError on a mismatch, so the same checks run against the
real oracle (test_oracle_pins.py) and against deliberately broken copies of
it (test_oracle_mutants.py).

None of these recomputes the oracle's arithmetic the oracle's way: the
references are direct inversion of the design matrix rebuilt from the
history, the Sherman-Morrison closed form of repeated updates, ridge least
squares, an exact rational hand derivation, explicit loops for argmax and
pruning, and statistical convergence on a known linear reward.
"""
import math

import numpy as np

from oracle import Oracle


def _rand_contexts(rng, T, B, d):
    x = rng.standard_normal((T, B, d))
    x[:, :, 0] = 1.0
    return x


def _brute_scores(hist, lam, d, x, alpha):
    """Scores of one arm from its history via direct inversion / solve."""
    A = lam * np.eye(d)
    b = np.zeros(d)
    for xs, rs in hist:
        A += np.outer(xs, xs)
        b += rs * xs
    theta = np.linalg.solve(A, b)
    quad = float(x @ np.linalg.solve(A, x))
    w = math.sqrt(max(0.0, quad))
    return A, b, theta, theta @ x + alpha * w, theta @ x - alpha * w


def _brute_trajectory(lib, B, K, d, T, lam, alpha0, sched, prune, period, seed, sticky=True):
    """Drive the oracle with random contexts and rewards and check every
    decision against brute force (explicit history, np.linalg, plain loops).
    sticky=False: rule 1 re-evaluated at each of its steps over every arm.
    Returns the number of arms that came back after rule 1 removed them."""
    rng = np.random.default_rng(seed)
    xs = _rand_contexts(rng, T, B, d)
    rs = rng.uniform(-2.0, 0.0, size=(T, B))
    ora = Oracle(B, K, d, lam, alpha0, sched, prune, period, lib=lib)
    if not sticky:
        ora.set_sticky(False)
    hist = [[[] for _ in range(K)] for _ in range(B)]
    active = np.ones((B, K), dtype=bool)
    returned = 0
    r_prev = None
    for t in range(T):
        ucb, lcb, keep, action = ora.decide(xs[t], r_prev)
        alpha = alpha0 if sched == 0 else alpha0 / math.sqrt(t + 1.0)
        prune_step = prune and t > 0 and t % period == 0
        for i in range(B):
            scored = active[i] | (prune_step and not sticky)
            U = np.full(K, -np.inf)
            L = np.full(K, -np.inf)
            for k in range(K):
                if scored[k]:
                    _, _, _, U[k], L[k] = _brute_scores(hist[i][k], lam, d, xs[t, i], alpha)
            for k in range(K):
                if scored[k]:
                    assert abs(ucb[i, k] - U[k]) <= 1e-9 * max(1.0, abs(U[k])), (t, i, k)
                    assert abs(lcb[i, k] - L[k]) <= 1e-9 * max(1.0, abs(L[k])), (t, i, k)
                else:
                    assert ucb[i, k] == -np.inf
            new_active = active[i].copy()
            if prune_step:
                lstar = max(L[k] for k in range(K) if scored[k])
                for k in range(K):
                    if scored[k]:
                        new_active[k] = not U[k] < lstar
                returned += int((new_active & ~active[i]).sum())
            assert (keep[i] == new_active).all(), (t, i)
            best = -1
            for k in range(K):
                if new_active[k] and (best < 0 or U[k] > U[best]):
                    best = k
            assert action[i] == best, (t, i, action[i], best)
            active[i] = new_active
            hist[i][best].append((xs[t, i], rs[t, i]))
        ora.commit(xs[t], action, keep)
        r_prev = rs[t]
    ora.flush(r_prev)
    for i in range(B):
        st = ora.get(i)
        for k in range(K):
            A, b, theta, _, _ = _brute_scores(hist[i][k], lam, d, xs[0, i], 0.0)
            assert np.allclose(st["A"][k], A, rtol=1e-12, atol=1e-12)
            assert np.allclose(st["b"][k], b, rtol=1e-12, atol=1e-12)
            Ainv = np.linalg.inv(A)
            assert np.abs(st["Ainv"][k] - Ainv).max() <= 1e-10 * np.abs(Ainv).max()
            assert np.abs(st["theta"][k] - theta).max() <= 1e-10 * max(1.0, np.abs(theta).max())
            assert st["nsel"][k] == len(hist[i][k])
        assert (st["active"] == active[i]).all()
    return returned


def pin_brute_force_small(lib):
    """Direct inversion + explicit argmax/prune loops on tiny random cases."""
    _brute_trajectory(lib, B=2, K=3, d=1, T=30, lam=1.0, alpha0=1.0, sched=0, prune=0,
                      period=5, seed=1)
    _brute_trajectory(lib, B=2, K=4, d=2, T=40, lam=0.5, alpha0=0.7, sched=1, prune=1,
                      period=7, seed=2)
    _brute_trajectory(lib, B=3, K=4, d=4, T=48, lam=2.0, alpha0=0.5, sched=0, prune=1,
                      period=5, seed=3)
    _brute_trajectory(lib, B=1, K=4, d=8, T=64, lam=1.0, alpha0=0.3, sched=0, prune=1,
                      period=4, seed=4)


def pin_nonsticky_rule_one(lib):
    """Rule 1 re-evaluated at each of its steps (the non-sticky reading):
    the kept set is recomputed from every arm with that step's scores, so an
    arm removed at one step can come back at a later one; the same brute
    force as above, also with the refinement's moving action space."""
    n = _brute_trajectory(lib, B=3, K=6, d=2, T=80, lam=1.0, alpha0=0.8, sched=0, prune=1,
                          period=4, seed=31, sticky=False)
    n += _brute_trajectory(lib, B=2, K=5, d=4, T=60, lam=0.5, alpha0=1.5, sched=1, prune=1,
                           period=3, seed=32, sticky=False)
    assert n > 0, "no removed arm came back"
    _brute_refine_trajectory(lib, B=2, K=14, d=2, T=60, stride=3, half=2, period=5, mature=20,
                             min_n=2, prune=1, pperiod=3, seed=33, sticky=False)
    # once exploiting, rule 1 no longer runs: the kept set stands at its steps
    e = Oracle(1, 6, 2, 1.0, 0.1, 0, 1, 4, lib=lib)
    e.set_sticky(False)
    e.set_exploit(True, ph_delta=0.05, ph_lambda=1e9, ph_window=10, ph_min_rounds=10)
    rng = np.random.default_rng(36)
    xs = _rand_contexts(rng, 40, 1, 2)
    r = None
    kept = None
    for t in range(40):
        u, l, k, a = e.step(xs[t], r)
        if t == 9:
            assert k[0].sum() == 2                 # rule 1 removed arms while exploring
        if t >= 10:
            assert np.array_equal(u, l)            # Eq. 2 scores
            kept = k[0] if kept is None else kept
            assert np.array_equal(k[0], kept), t   # and no rule-1 step touches the set
        r = rng.uniform(-2.0, 0.0, size=1)
    # up to the first rule-1 step both readings coincide
    a = Oracle(2, 5, 2, 1.0, 0.8, 0, 1, 6, lib=lib)
    b = Oracle(2, 5, 2, 1.0, 0.8, 0, 1, 6, lib=lib)
    b.set_sticky(False)
    rng = np.random.default_rng(34)
    xs = _rand_contexts(rng, 7, 2, 2)
    r = None
    for t in range(7):
        ua, _, ka, aa = a.step(xs[t], r)
        ub, _, kb, ab = b.step(xs[t], r)
        assert np.array_equal(ua, ub) and np.array_equal(ka, kb) and np.array_equal(aa, ab), t
        r = rng.uniform(-2.0, 0.0, size=2)


def pin_repeated_update_closed_form(lib):
    """n identical updates with x: the Sherman-Morrison closed form.

    A = lam I + n x x^T  =>  A^{-1} = (I - n x x^T / (lam + n |x|^2)) / lam,
    x^T A^{-1} x = |x|^2 / (lam + n |x|^2),  theta = (sum r) x / (lam + n |x|^2).
    """
    d, lam, n = 5, 1.7, 37
    x = np.array([1.0, -0.5, 2.0, 0.25, -1.5])
    rng = np.random.default_rng(5)
    rs = rng.normal(size=n)
    ora = Oracle(1, 1, d, lam, 0.8, 0, 0, 50, lib=lib)
    r_prev = None
    for s in range(n):
        ucb, lcb, keep, action = ora.step(x[None, :], r_prev)
        assert action[0] == 0
        r_prev = rs[s:s + 1]
    ucb, lcb, keep, action = ora.decide(x[None, :], r_prev)
    nx2 = float(x @ x)
    denom = lam + n * nx2
    Ainv = (np.eye(d) - n * np.outer(x, x) / denom) / lam
    theta = rs.sum() * x / denom
    st = ora.get(0)
    assert np.abs(st["Ainv"][0] - Ainv).max() <= 1e-12
    assert np.abs(st["theta"][0] - theta).max() <= 1e-12
    w = math.sqrt(nx2 / denom)
    m = rs.sum() * nx2 / denom
    assert abs(ucb[0, 0] - (m + 0.8 * w)) <= 1e-12
    assert abs(lcb[0, 0] - (m - 0.8 * w)) <= 1e-12


def pin_ridge_least_squares(lib):
    """K = 1: theta is the ridge solution of the observed (x, r) pairs (Eq. 5)."""
    d, lam, T = 6, 0.3, 80
    rng = np.random.default_rng(6)
    xs = _rand_contexts(rng, T, 1, d)[:, 0]
    rs = rng.normal(size=T)
    ora = Oracle(1, 1, d, lam, 0.0, 0, 0, 50, lib=lib)
    r_prev = None
    for t in range(T):
        ora.step(xs[t][None, :], r_prev)
        r_prev = rs[t:t + 1]
    ora.flush(r_prev)
    Xa = np.vstack([xs, math.sqrt(lam) * np.eye(d)])
    ya = np.concatenate([rs, np.zeros(d)])
    theta_ls = np.linalg.lstsq(Xa, ya, rcond=None)[0]
    assert np.abs(ora.get(0)["theta"][0] - theta_ls).max() <= 1e-10


def pin_rational_worked_example(lib):
    """Hand-worked d = 2, K = 2 trajectory in exact rational arithmetic."""
    from golden_example import load_worked_example
    ex = load_worked_example()
    d, K = 2, 2
    lam, alpha = ex["lambda"], ex["alpha"]
    ora = Oracle(1, K, d, float(lam), float(alpha), 0, 0, 50, lib=lib)
    r_prev = None
    for step in ex["steps"]:
        x = np.array([float(v) for v in step["x"]])
        ucb, lcb, keep, action = ora.step(x[None, :], r_prev)
        assert action[0] == step["action"], (step, action)
        for k in range(K):
            m, q = step["mean"][k], step["quad"][k]
            expect = float(m) + float(alpha) * math.sqrt(float(q))
            assert abs(ucb[0, k] - expect) <= 1e-13, (step, k, ucb[0, k], expect)
        r_prev = np.array([float(step["reward"])])
    ora.flush(r_prev)
    st = ora.get(0)
    for k, (Ainv, theta) in enumerate(zip(ex["final_Ainv"], ex["final_theta"])):
        assert np.abs(st["Ainv"][k] - np.array(Ainv, dtype=float)).max() <= 1e-14
        assert np.abs(st["theta"][k] - np.array(theta, dtype=float)).max() <= 1e-14


def pin_textbook_reductions(lib):
    """K = 1 always picks arm 0; untouched arms tie and are swept in index
    order; alpha = 0 is greedy on theta^T x; d = 1 is the scalar formula."""
    rng = np.random.default_rng(7)
    ora = Oracle(2, 1, 3, 1.0, 1.0, 0, 1, 5, lib=lib)
    r_prev = None
    for t in range(20):
        x = _rand_contexts(rng, 1, 2, 3)[0]
        _, _, _, action = ora.step(x, r_prev)
        assert (action == 0).all()
        r_prev = rng.normal(size=2)
    K = 6
    ora = Oracle(1, K, 4, 1.0, 1.0, 0, 0, 50, lib=lib)
    r_prev = None
    seen = []
    x = _rand_contexts(rng, 1, 1, 4)[0]
    for t in range(K):
        # a touched arm now has mean r |x|^2/(lam+|x|^2) < 0 and a smaller width
        ucb, _, _, action = ora.step(x, r_prev)
        seen.append(int(action[0]))
        r_prev = np.array([-1.0])
    assert seen == list(range(K))
    ora = Oracle(1, 3, 2, 1.0, 0.0, 0, 0, 50, lib=lib)
    hist = [[] for _ in range(3)]
    r_prev = None
    for t in range(30):
        x = np.array([1.0, rng.normal()])
        ucb, _, _, action = ora.step(x[None, :], r_prev)
        greedy = []
        for k in range(3):
            A = np.eye(2) + sum((np.outer(a, a) for a, _ in hist[k]), np.zeros((2, 2)))
            b = sum((r * a for a, r in hist[k]), np.zeros(2))
            greedy.append(np.linalg.solve(A, b) @ x)
        best = max(range(3), key=lambda k: (greedy[k], -k))
        assert action[0] == best
        r = float(rng.normal() - 0.3 * best)
        hist[best].append((x, r))
        r_prev = np.array([r])
    lam, alpha = 2.0, 0.6
    ora = Oracle(1, 2, 1, lam, alpha, 0, 0, 50, lib=lib)
    sums = [[lam, 0.0], [lam, 0.0]]   # per arm: lam + sum x^2, sum r x
    r_prev = None
    for t in range(25):
        x = float(rng.uniform(0.5, 2.0))
        ucb, _, _, action = ora.step(np.array([[x]]), r_prev)
        for k in range(2):
            a, s = sums[k]
            assert abs(ucb[0, k] - (s / a * x + alpha * abs(x) / math.sqrt(a))) <= 1e-12
        r = float(rng.normal())
        sums[action[0]][0] += x * x
        sums[action[0]][1] += r * x
        r_prev = np.array([r])


def pin_prune_invariants(lib):
    """Along random trajectories with pruning: the action set only shrinks,
    the arms with the largest UCB and the largest LCB always survive, so the
    set is never empty; with alpha = 0 one prune leaves only the arms whose
    estimate ties the best."""
    rng = np.random.default_rng(8)
    B, K, d, T = 4, 12, 4, 120
    ora = Oracle(B, K, d, 1.0, 0.4, 0, 1, 10, lib=lib)
    prev = np.ones((B, K), dtype=bool)
    r_prev = None
    for t in range(T):
        x = _rand_contexts(rng, 1, B, d)[0]
        ucb, lcb, keep, action = ora.step(x, r_prev)
        assert not (keep & ~prev).any()
        assert keep.any(axis=1).all()
        if t > 0 and t % 10 == 0:
            for i in range(B):
                act = np.flatnonzero(prev[i])
                assert keep[i, act[np.argmax(ucb[i, act])]]
                assert keep[i, act[np.argmax(lcb[i, act])]]
        prev = keep
        r_prev = rng.normal(size=B) - 0.1 * action
    ora = Oracle(1, 5, 2, 1.0, 0.0, 0, 1, 6, lib=lib)
    r_prev = None
    for t in range(7):
        x = np.array([[1.0, 0.5]])
        ucb, lcb, keep, action = ora.step(x, r_prev)
        r_prev = np.array([-1.0 - 0.1 * t])
    # alpha = 0: UCB = LCB = theta^T x, so the prune at t = 6 keeps exactly
    # the arms whose estimate equals the maximum
    m = ucb[0]
    assert keep[0].sum() == (m == m.max()).sum()
    assert keep[0, int(np.argmax(m))]


def pin_convergence_linear_reward(lib):
    """Linear rewards r = theta*_k^T x + N(0, s^2): the estimates converge at
    the statistical rate and the tuner settles on the best arm."""
    rng = np.random.default_rng(9)
    K, d, T, s = 3, 4, 6000, 0.1
    theta_star = np.array([[0.0, 0.5, -0.3, 0.2],
                           [0.4, 0.5, -0.3, 0.2],
                           [0.1, -0.2, 0.3, 0.0]])
    ora = Oracle(1, K, d, 1.0, 0.5, 0, 0, 50, lib=lib)
    r_prev = None
    best_count = 0
    regret = np.zeros(T)
    for t in range(T):
        x = np.concatenate([[1.0], rng.standard_normal(d - 1)])
        _, _, _, action = ora.step(x[None, :], r_prev)
        a = int(action[0])
        means = theta_star @ x
        regret[t] = means.max() - means[a]
        if t >= T - 1000 and a == int(np.argmax(means)):
            best_count += 1
        r_prev = np.array([means[a] + s * rng.standard_normal()])
    ora.flush(r_prev)
    st = ora.get(0)
    n1 = st["nsel"][1]
    err = np.linalg.norm(st["theta"][1] - theta_star[1])
    assert n1 > T // 2
    assert err <= 5 * s * math.sqrt(d / n1) + np.linalg.norm(theta_star[1]) / n1
    assert best_count >= 900
    assert regret[T // 2:].sum() < regret[:T // 2].sum()


ALL_PINS = [pin_brute_force_small, pin_nonsticky_rule_one, pin_repeated_update_closed_form, pin_ridge_least_squares,
            pin_rational_worked_example, pin_textbook_reductions, pin_prune_invariants,
            pin_convergence_linear_reward]


# ---- the paper's pruning heuristics (rule bits 2, 4, 8; Sec. 4.3) ----

def _scripted(lib, K, d, rule, heur, plan, x=None, lam=1.0, alpha=1.0):
    """Drive one oracle instance with scripted actions and rewards.

    plan: list of (action, reward); the action is committed whatever the
    oracle proposes, so each arm's reward history is exactly the script.
    Returns the decide() outputs of every step and the oracle."""
    ora = Oracle(1, K, d, lam, alpha, 0, rule, 1000, lib=lib)
    ora.set_heuristics(**heur)
    x = np.ones((1, d)) if x is None else x
    r_prev = None
    outs = []
    for a, r in plan:
        ucb, lcb, keep, action, marg = ora.decide(x, r_prev, margins=True)
        outs.append((ucb[0], keep[0], marg[0]))
        ora.commit(x, np.array([a]), keep)
        r_prev = np.array([r])
    ucb, lcb, keep, action, marg = ora.decide(x, r_prev, margins=True)
    outs.append((ucb[0], keep[0], marg[0]))
    return outs, ora


HEUR = dict(ext_rounds=60, ext_min_n=3, ext_thr=-1.2, hist_after=30, hist_min_n=6, hist_kappa=1.0,
            hist_min_arms=3, cascade_k=0)


def pin_extreme_pruning(lib):
    """Sec. 4.3 extreme pruning: within the first 60 rounds an arm with at
    least 3 rewards averaging below -1.2 leaves for good; 2 rewards are not
    enough, a mean at -1.1 stays, and after round 60 the rule is off."""
    plan = [(1, -1.5), (1, -1.4), (1, -1.6),      # arm 1: n = 3, mean -1.5
            (2, -1.1), (2, -1.1), (2, -1.1),      # arm 2: n = 3, mean -1.1
            (3, -5.0), (3, -5.0)]                 # arm 3: n = 2
    outs, ora = _scripted(lib, 5, 2, 2, HEUR, plan)
    ucb, keep, marg = outs[-1]
    assert list(keep) == [True, False, True, True, True]
    assert ucb[1] == -np.inf and np.isfinite(ucb[3])
    assert marg[1] == np.inf and abs(marg[2] - 0.1) < 1e-12 and marg[3] == np.inf
    assert abs(outs[3][2][1] - 0.3) < 1e-12      # judged at step 3, gone afterwards
    # arm 1 leaves at the decision after its third reward (step 3), not before
    assert outs[2][1][1] and not outs[3][1][1]
    # the third reward lands at round 59 (judged) or round 60 (too late)
    outs, _ = _scripted(lib, 5, 2, 2, HEUR, [(0, -1.0)] * 56 + [(4, -2.0)] * 3)
    assert not outs[-1][1][4]
    outs, _ = _scripted(lib, 5, 2, 2, HEUR, [(0, -1.0)] * 57 + [(4, -2.0)] * 3)
    assert outs[-1][1][4]


def pin_historical_pruning(lib):
    """Sec. 4.3 historical pruning, worked by hand: qualifying arms' mean
    rewards -1, -1.1, -2, -1.05 have mean -1.2875 and population standard
    deviation 0.41288; only the arm 1.0 below the best is more than one
    deviation worse.  With too few qualifying arms nothing is compared."""
    heur = dict(HEUR, hist_after=0, hist_min_n=1, hist_min_arms=4)
    plan = [(0, -1.0), (1, -1.1), (2, -2.0), (3, -1.05)]
    outs, _ = _scripted(lib, 5, 2, 4, heur, plan)
    ucb, keep, marg = outs[-1]
    assert list(keep) == [True, True, False, True, True]
    sigma = 0.41288
    assert abs(marg[2] - (1.0 - sigma)) < 1e-5 and abs(marg[0] - sigma) < 1e-5
    outs, _ = _scripted(lib, 5, 2, 4, heur, plan[:2])
    assert outs[-1][1].all()
    # hist_after: the rule waits for its round
    outs, _ = _scripted(lib, 5, 2, 4, dict(heur, hist_after=10), plan)
    assert outs[-1][1].all()


def pin_cascade_pruning(lib):
    """Sec. 4.3 cascade: an arm pruned below half of the top clock (index <
    cascade_k) takes every lower arm with it; one above does not."""
    heur = dict(HEUR, cascade_k=4)
    plan = [(2, -2.0)] * 3 + [(1, -0.5)] * 3
    outs, _ = _scripted(lib, 6, 2, 2 | 8, heur, plan)
    assert list(outs[3][1]) == [False, False, False, True, True, True]
    plan = [(4, -2.0)] * 3
    outs, _ = _scripted(lib, 6, 2, 2 | 8, heur, plan)
    assert list(outs[-1][1]) == [True, True, True, True, False, True]


def pin_heuristics_keep_one_arm(lib):
    """If the rules would remove every arm, the one with the best mean reward
    stays: arm 2 fails the extreme rule and its cascade takes arms 0 and 1
    (cascade_k = 3); arm 1's mean, -0.4, is the best."""
    plan = [(0, -0.5), (1, -0.4)] + [(2, -2.0)] * 3
    outs, _ = _scripted(lib, 3, 2, 2 | 8, dict(HEUR, cascade_k=3), plan)
    assert list(outs[-1][1]) == [False, True, False]


def pin_heuristics_brute_force(lib):
    """Random scripted histories against an independent restatement of the
    rules (numpy, vectorised), step by step."""
    rng = np.random.default_rng(11)
    for trial in range(6):
        K = int(rng.integers(4, 12))
        heur = dict(ext_rounds=int(rng.integers(5, 40)), ext_min_n=int(rng.integers(1, 4)),
                    ext_thr=float(rng.uniform(-1.6, -0.9)), hist_after=int(rng.integers(0, 30)),
                    hist_min_n=int(rng.integers(1, 5)), hist_kappa=float(rng.uniform(0.3, 2.0)),
                    hist_min_arms=int(rng.integers(2, 5)), cascade_k=int(rng.integers(0, K)))
        rule = int(rng.choice([2, 4, 8 | 2, 8 | 4, 14]))
        ora = Oracle(1, K, 3, 1.0, 0.7, 0, rule, 1000, lib=lib)
        ora.set_heuristics(**heur)
        n = np.zeros(K, int)
        s = np.zeros(K)
        active = np.ones(K, bool)
        x = np.array([[1.0, 0.3, -0.2]])
        r_prev = None
        for t in range(50):
            ucb, lcb, keep, action = ora.decide(x, r_prev)
            mean = np.where(n > 0, s / np.maximum(n, 1), 0.0)
            gone = np.zeros(K, bool)
            if rule & 2 and t < heur["ext_rounds"]:
                gone |= active & (n >= heur["ext_min_n"]) & (mean < heur["ext_thr"])
            q = active & (n >= heur["hist_min_n"])
            if rule & 4 and t >= heur["hist_after"] and q.sum() >= heur["hist_min_arms"]:
                sig = mean[q].std()
                gone |= q & (mean[q].max() - mean > heur["hist_kappa"] * sig)
            if rule & 8:
                low = np.flatnonzero(gone & (np.arange(K) < heur["cascade_k"]))
                if low.size:
                    gone |= np.arange(K) < low.max()
            stay = active & ~gone
            if not stay.any():
                cand = np.flatnonzero(active)
                scored = [k for k in cand if n[k] > 0]
                stay[max(scored, key=lambda k: (mean[k], -k)) if scored else cand[0]] = True
            assert np.array_equal(keep[0], stay), (trial, t)
            a = int(rng.choice(np.flatnonzero(stay)))
            r = float(rng.normal(-1.2, 0.5))
            ora.commit(x, np.array([a]), keep)
            n[a] += 1
            s[a] += r
            active = stay
            r_prev = np.array([r])


ALL_PINS += [pin_extreme_pruning, pin_historical_pruning, pin_cascade_pruning,
             pin_heuristics_keep_one_arm, pin_heuristics_brute_force]


# ---- Page-Hinkley switch to greedy exploitation (Sec. 4.2, Eq. 2) ----

PH = dict(ph_delta=0.05, ph_lambda=5.0, ph_window=100, ph_min_rounds=100)


def _ph_by_definition(rewards, delta, lam):
    """Alarm rounds of the two-sided Page-Hinkley test computed from its
    definition: after each restart, the cumulative sums are rebuilt from the
    rewards seen since then, each running mean recomputed from scratch
    (reward s enters at round s + 1)."""
    alarms, seg = [], []
    for s, r in enumerate(rewards):
        seg.append(float(r))
        up = dn = up_min = dn_min = 0.0
        for q in range(len(seg)):
            rbar = sum(seg[:q + 1]) / (q + 1)
            up += seg[q] - rbar - delta
            dn += rbar - seg[q] - delta
            up_min, dn_min = min(up_min, up), min(dn_min, dn)
        if max(up - up_min, dn - dn_min) > lam:
            alarms.append(s + 1)
            seg = []
    return alarms


def _run_rewards(lib, rewards, K=3, d=2, ph=PH, rule=0, x_fn=None):
    """One instance: the oracle picks its own arms, the reward of every pick
    is scripted; returns per-round (ucb, lcb, action) and the oracle."""
    ora = Oracle(1, K, d, 1.0, 1.0, 0, rule, 50, lib=lib)
    ora.set_exploit(True, **ph)
    rng = np.random.default_rng(3)
    r_prev = None
    hist = []
    for t, r in enumerate(rewards):
        x = x_fn(t, rng) if x_fn else np.concatenate([[1.0], rng.standard_normal(d - 1)])[None, :]
        ucb, lcb, keep, action = ora.step(x, r_prev)
        hist.append((x[0], ucb[0], lcb[0], int(action[0])))
        r_prev = np.array([r])
    return hist, ora


def pin_page_hinkley_worked_example(lib):
    """The hand-worked example under tests/golden/ (exact rationals): the
    test's state, margin, alarm rounds and switch round after every round,
    an upward and a downward alarm with a restart after each, and no test
    once exploiting."""
    from golden_example import load_page_hinkley_example
    ex = load_page_hinkley_example()
    ora = Oracle(1, 2, 2, 1.0, 1.0, 0, 0, 50, lib=lib)
    ora.set_exploit(True, ph_delta=float(ex["delta"]), ph_lambda=float(ex["lambda"]),
                    ph_window=ex["window"], ph_min_rounds=ex["min_rounds"])
    x = np.array([[1.0, 0.5]])
    rewards = {rd["t"] - 1: float(rd["r"]) for rd in ex["rounds"]}
    ora.step(x, None)
    last = 0
    for rd in ex["rounds"]:
        t = rd["t"]
        ora.step(x, np.array([rewards[t - 1]]))
        stats, margin, got_last, mode = ora.page_hinkley(0)
        want = np.array([float(v) for v in rd["state"]])
        assert np.allclose(stats, want, rtol=0, atol=1e-12), (t, stats, want)
        assert abs(margin - float(rd["margin"])) <= 1e-12, (t, margin)
        if rd["alarm"]:
            last = t
        assert got_last == last and mode == rd["mode"], (t, got_last, mode)


def pin_page_hinkley_threshold_is_strict(lib):
    """The test alarms when its statistic exceeds lambda, not when it reaches
    it: with delta = 0 and lambda = 1, rewards 0, 2 bring m+ to exactly 1
    (binary-exact) with no alarm; a further 2 brings it to 5/3 and alarms."""
    hist, ora = _run_rewards(lib, [0.0, 2.0, 2.0, 2.0],
                             ph=dict(ph_delta=0.0, ph_lambda=1.0, ph_window=50, ph_min_rounds=50))
    # _run_rewards feeds reward s at round s + 1 and stops after the last
    # decision, so the last reward is never fed: rounds 1..3 have run
    stats, margin, last, mode = ora.page_hinkley(0)
    assert last == 3 and np.all(stats == 0.0), (last, stats)
    hist, ora = _run_rewards(lib, [0.0, 2.0, 0.0],
                             ph=dict(ph_delta=0.0, ph_lambda=1.0, ph_window=50, ph_min_rounds=50))
    stats, margin, last, mode = ora.page_hinkley(0)
    assert last == 0 and margin == 0.0 and stats[2] == 1.0 and stats[3] == 0.0, (last, margin, stats)


def pin_page_hinkley_switch_round(lib):
    """A stationary reward sequence never alarms, so exploitation starts at
    round max(min_rounds, window); a step of height h after s0 constant
    rewards raises the upward statistic by h*s0/(s0+q) - delta at the q-th
    round after it (the running mean moves by h/(s0+q) per round), so the
    alarm comes at the first k whose partial sum exceeds lambda, and the
    switch is postponed to that round plus the window; on noise, the alarm
    rounds are those of the test's definition recomputed from scratch."""
    flat = [-1.0] * 160
    hist, ora = _run_rewards(lib, flat)
    assert ora.page_hinkley(0)[3] == 100
    assert all(h[1][h[3]] != h[2][h[3]] for h in hist[:100])       # UCB > LCB while exploring
    hist, ora = _run_rewards(lib, flat, ph=dict(PH, ph_min_rounds=130))
    assert ora.page_hinkley(0)[3] == 130
    s0, h, delta, lam = 80, 0.8, PH["ph_delta"], PH["ph_lambda"]
    acc, k = 0.0, 0
    while acc <= lam:
        k += 1
        acc += h * s0 / (s0 + k) - delta
    step = [-1.0] * s0 + [-1.0 + h] * 200
    hist, ora = _run_rewards(lib, step)
    _, _, last, mode = ora.page_hinkley(0)
    assert last == s0 + k and mode == last + PH["ph_window"], (last, mode, s0 + k)
    noisy = list(np.random.default_rng(4).normal(-1.0, 0.4, 400))
    hist, ora = _run_rewards(lib, noisy)
    alarms = _ph_by_definition(noisy, PH["ph_delta"], PH["ph_lambda"])
    _, _, last, mode = ora.page_hinkley(0)
    before = [a for a in alarms if mode < 0 or a <= mode]
    assert last == (before[-1] if before else 0), (last, before)
    assert len(alarms) >= 2


def pin_greedy_after_switch(lib):
    """Once exploiting, the choice is argmax theta_k^T x_t over the active arms
    (Eq. 2, ties to the lowest index), reported as both UCB and LCB, with
    theta_k recomputed from the arm's history by direct solve."""
    K, d = 4, 3
    rng = np.random.default_rng(21)
    ora = Oracle(1, K, d, 1.0, 1.0, 0, 0, 50, lib=lib)
    ora.set_exploit(True, ph_delta=0.05, ph_lambda=1e9, ph_window=10, ph_min_rounds=10)
    hist = [[] for _ in range(K)]
    r_prev = None
    for t in range(40):
        x = np.concatenate([[1.0], rng.standard_normal(d - 1)])
        ucb, lcb, keep, action = ora.step(x[None, :], r_prev)
        a = int(action[0])
        if t >= 10:
            m = []
            for k in range(K):
                A = np.eye(d) + sum((np.outer(z, z) for z, _ in hist[k]), np.zeros((d, d)))
                b = sum((q * z for z, q in hist[k]), np.zeros(d))
                m.append(np.linalg.solve(A, b) @ x)
            assert np.allclose(ucb[0], m, atol=1e-12) and np.allclose(lcb[0], m, atol=1e-12)
            assert a == max(range(K), key=lambda k: (m[k], -k))
        r = float(rng.normal(-1.0 + 0.2 * a, 0.1))
        hist[a].append((x, r))
        r_prev = np.array([r])


ALL_PINS += [pin_page_hinkley_worked_example, pin_page_hinkley_threshold_is_strict,
             pin_page_hinkley_switch_round, pin_greedy_after_switch]


# ---- mixed-maturity refinement of the action space (Sec. 4.4) ----

def _in_space(k, lo, hi, stride):
    return lo <= k <= hi and (hi - k) % stride == 0


def _brute_refine_trajectory(lib, B, K, d, T, stride, half, period, mature, min_n, prune, pperiod,
                             seed, alpha0=0.6, sticky=True):
    """Drive the oracle with refinement on and check every step against an
    independent restatement: the action space as an explicit set, scores by
    direct solve from each arm's full history (models persist while an arm is
    outside the space), rule 1, the argmax, and the anchor chosen after the
    decision (best mean reward with enough samples before maturity, the
    decision itself after).  sticky=False: rule 1 re-evaluated at each of its
    steps over the whole action space.  Returns the number of arms that
    re-entered the space with a history of their own."""
    rng = np.random.default_rng(seed)
    xs = _rand_contexts(rng, T, B, d)
    rs = rng.uniform(-2.0, 0.0, size=(T, B))
    ora = Oracle(B, K, d, 1.0, alpha0, 0, prune, pperiod, lib=lib)
    ora.set_refine(True, period, stride, half, mature, min_n)
    if not sticky:
        ora.set_sticky(False)
    hist = [[[] for _ in range(K)] for _ in range(B)]
    pruned = np.zeros((B, K), dtype=bool)
    win = [(0, K - 1, stride) for _ in range(B)]
    seen_out = np.zeros((B, K), dtype=bool)
    reentries = 0
    r_prev = None
    for t in range(T):
        ucb, lcb, keep, action = ora.decide(xs[t], r_prev)
        for i in range(B):
            lo, hi, st = win[i]
            reeval = prune and t > 0 and t % pperiod == 0 and not sticky
            space = [k for k in range(K) if _in_space(k, lo, hi, st) and (reeval or not pruned[i, k])]
            for k in range(K):
                if k in space:
                    if seen_out[i, k] and hist[i][k]:
                        reentries += 1
                        seen_out[i, k] = False
                    _, _, _, U, L = _brute_scores(hist[i][k], 1.0, d, xs[t, i], alpha0)
                    assert abs(ucb[i, k] - U) <= 1e-9 * max(1.0, abs(U)), (t, i, k)
                    assert abs(lcb[i, k] - L) <= 1e-9 * max(1.0, abs(L)), (t, i, k)
                else:
                    assert ucb[i, k] == -np.inf, (t, i, k)
                    seen_out[i, k] = True
            survivors = list(space)
            if prune and t > 0 and t % pperiod == 0:
                lstar = max(lcb[i, k] for k in space)
                survivors = [k for k in space if not ucb[i, k] < lstar]
                if reeval:
                    pruned[i] = False
                for k in space:
                    if k not in survivors:
                        pruned[i, k] = True
            assert (keep[i] == ~pruned[i]).all(), (t, i)
            best = max(survivors, key=lambda k: (ucb[i, k], -k))
            assert action[i] == best, (t, i, action[i], best)
            hist[i][best].append((xs[t, i], rs[t, i]))
            if t > 0 and t % period == 0:
                if t < mature:
                    # the means count the rewards folded in so far, not this step's
                    means = {k: sum(q for _, q in hist[i][k][:len(hist[i][k]) - (k == best)])
                             / (len(hist[i][k]) - (k == best)) for k in survivors
                             if len(hist[i][k]) - (k == best) >= min_n}
                    anchor = max(means, key=lambda k: (means[k], -k)) if means else None
                else:
                    anchor = best
                if anchor is not None:
                    win[i] = (max(0, anchor - half), min(K - 1, anchor + half), 1)
        ora.commit(xs[t], action, keep)
        for i in range(B):
            assert ora.window(i) == win[i], (t, i, ora.window(i), win[i])
        r_prev = rs[t]
    return reentries


def pin_refinement_brute_force(lib):
    """Refinement with coarse grids, moving windows, rule 1 and re-entering
    arms, against the explicit restatement above."""
    n = _brute_refine_trajectory(lib, B=2, K=12, d=2, T=60, stride=3, half=2, period=4, mature=20,
                                 min_n=2, prune=1, pperiod=7, seed=11)
    n += _brute_refine_trajectory(lib, B=2, K=20, d=3, T=70, stride=4, half=1, period=3, mature=30,
                                  min_n=1, prune=0, pperiod=5, seed=12)
    n += _brute_refine_trajectory(lib, B=1, K=9, d=4, T=50, stride=2, half=3, period=5, mature=10,
                                  min_n=3, prune=1, pperiod=4, seed=13)
    assert n > 0, "no arm re-entered the action space with a history"


def pin_refinement_coarse_sweep(lib):
    """Untouched arms tie exactly, so the first decisions sweep the coarse grid
    in index order; the grid is counted down from the top arm."""
    K, d = 40, 2
    ora = Oracle(1, K, d, 1.0, 1.0, 0, 0, 50, lib=lib)
    ora.set_refine(True, 100, 10, 10, 100, 4)
    x = np.array([[1.0, 0.5]])
    acts = []
    r_prev = None
    for t in range(4):
        ucb, lcb, keep, action = ora.decide(x, r_prev)
        if t == 0:
            assert np.isfinite(ucb[0]).sum() == 4
        acts.append(int(action[0]))
        ora.commit(x, action, keep)
        r_prev = np.array([-1.0])
    assert acts == [9, 19, 29, 39], acts


def pin_refinement_statistical_then_predictive(lib):
    """A scripted reward that depends only on the arm: before maturity the
    window centres on the coarse arm with the best mean reward once it has
    enough samples; at maturity it centres on that step's choice."""
    K, d = 60, 2
    ora = Oracle(1, K, d, 1.0, 0.0, 0, 0, 50, lib=lib)      # alpha = 0: greedy on theta
    ora.set_refine(True, 10, 10, 4, 30, 2)
    reward = lambda k: -1.0 - abs(k - 33) / 20.0      # best coarse arm: 29 (grid 9, 19, ..., 59)
    x = np.array([[1.0, 0.0]])
    r_prev = None
    for t in range(31):
        ucb, lcb, keep, action = ora.decide(x, r_prev)
        a = int(action[0])
        ora.commit(x, action, keep)
        r_prev = np.array([reward(a)])
        if t == 10:
            st = ora.get(0)
            n, rsum = st["nsel"], st["rsum"]
            cand = [k for k in range(9, K, 10) if n[k] >= 2]
            assert 29 in cand
            assert ora.window(0) == (25, 33, 1)
        if t == 30:
            assert ora.window(0) == (max(0, a - 4), min(K - 1, a + 4), 1)


def pin_refinement_skips_pruned_arms(lib):
    """The statistical anchor is taken among arms still in play: an arm that a
    cascade removed does not anchor the window, however good its mean."""
    K, d = 6, 2
    ora = Oracle(1, K, d, 1.0, 1.0, 0, 2 | 8, 50, lib=lib)
    ora.set_heuristics(ext_rounds=60, ext_min_n=1, ext_thr=-1.2, hist_after=1000, hist_min_n=100,
                       hist_kappa=1.0, hist_min_arms=3, cascade_k=4)
    ora.set_refine(True, 6, 1, 1, 100, 1)
    reward = {0: -1.0, 1: -0.5, 2: -1.0, 3: -3.0, 4: -1.0, 5: -1.0}
    x = np.array([[1.0, 0.0]])
    r_prev = None
    acts = []
    for t in range(7):
        ucb, lcb, keep, action = ora.decide(x, r_prev)
        acts.append(int(action[0]))
        ora.commit(x, action, keep)
        r_prev = np.array([reward[acts[-1]]])
    assert acts[:6] == [0, 1, 2, 3, 4, 5], acts
    assert list(keep[0]) == [0, 0, 0, 0, 1, 1]
    assert ora.window(0) == (3, 5, 1), ora.window(0)


ALL_PINS += [pin_refinement_brute_force, pin_refinement_coarse_sweep,
             pin_refinement_statistical_then_predictive, pin_refinement_skips_pruned_arms]
