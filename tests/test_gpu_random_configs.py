"""A seeded sweep of option combinations on the GPU against the oracle: the
context dimension (and with it the record layout), the arm count, the ridge
prior, the exploration schedule, the pruning rule bits, the switch to
exploitation and the refinement, drawn together so that combinations the
hand-written cases do not name are checked too.

Open loop (the same contexts and single-precision rewards to both sides),
with a reward change halfway so that switches and alarms both happen; every
score, prune bit, action, test state and action space is compared at every
step, and the final models through the export kernel."""
import numpy as np
import pytest

import parity
from gpu_helpers import compare_model, random_contexts, run_open_loop, say

pytestmark = pytest.mark.gpu


def _case(seed):
    rng = np.random.default_rng([2508, 1744, 99, seed])
    d = int(rng.choice([8, 16, 32]))
    K = int(rng.integers(1, 301 if d < 32 else 161))
    cfg = dict(B=int(rng.integers(1, 10)), K=K, d=d, lam=float(rng.choice([0.5, 1.0, 2.0])),
               alpha0=float(rng.uniform(0.0, 1.2)), sched=int(rng.integers(0, 2)),
               prune=int(rng.choice([0, 1, 3, 5, 13, 15])), period=int(rng.integers(5, 30)),
               heuristics=None)
    if cfg["prune"] & 14:
        # thresholds that fire within a 100-step run
        cfg["heuristics"] = dict(ext_rounds=40, ext_min_n=1, ext_thr=-1.0, hist_after=10, hist_min_n=2,
                                 hist_kappa=float(rng.uniform(0.3, 1.5)), hist_min_arms=3,
                                 cascade_k=int(rng.integers(0, K + 1)))
    if rng.random() < 0.5:
        cfg["exploit"] = dict(ph_delta=0.05, ph_lambda=5.0, ph_window=int(rng.integers(10, 40)),
                              ph_min_rounds=int(rng.integers(20, 60)))
    if K > 1 and rng.random() < 0.5:
        cfg["refine"] = dict(refine_period=int(rng.integers(5, 15)), refine_stride=int(rng.integers(2, 8)),
                             refine_half=int(rng.integers(0, 6)), refine_mature=int(rng.integers(10, 40)),
                             refine_min_n=int(rng.integers(1, 4)))
    return cfg


@pytest.mark.parametrize("seed", range(48))
def test_random_configuration(seed):
    cfg = _case(seed)
    T = 100
    X, R = random_contexts(9000 + seed, T, cfg["B"], cfg["d"])
    R[T // 2:, ::2] -= 1.0
    R = R.astype(np.float32).astype(np.float64)
    say(f"[random {seed}] {cfg}")
    a, m, s, tuner, rec = run_open_loop(cfg, X, R)
    st = parity.compare_open_loop(f"random {seed}", cfg, X, R, a, m, s, g_ph=rec["ph"], g_win=rec["win"])
    compare_model(tuner, st["oracle"], range(cfg["B"]), 1e-3, 1e-4)
    say(f"[random {seed}] max score err {st['max_score_err']:.2e}, forced {st['forced']}/{st['decisions']}, "
        f"greedy {st.get('greedy_decisions', 0)}, refinements {st.get('refinements', 0)}")
