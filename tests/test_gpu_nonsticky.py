"""The non-sticky reading of rule 1 on the GPU against the oracle: at each
rule-1 step the kept set is recomputed over the whole action space (every arm
of it scored), so arms removed at one step can come back at a later one.

Open loop over d = 8, 16, 32 and ragged arm counts, with the refinement's
moving action space and with the switch to exploitation; closed loop on the
three pruning workloads with rule 1 re-evaluated (cfg3n, cfg4n, cfg5n),
small with every instance and full size with probes."""
import numpy as np
import pytest
import torch

import parity
from agft_workloads import ENV, exogenous, get_workload, probe_instances
from gpu_helpers import compare_model, random_contexts, run_open_loop, say
from paper_2508_01744_amd import run_closed_loop

pytestmark = pytest.mark.gpu


def _returns(masks, K):
    """Arms whose mask bit came back on after being cleared, summed over instances."""
    keep = parity.mask_words_to_bool(masks, K)
    return int((keep[1:] & ~keep[:-1]).sum())


@pytest.mark.parametrize("d,K,period,alpha", [(8, 20, 5, 0.3), (16, 100, 7, 0.2), (32, 33, 4, 0.3),
                                              (16, 256, 6, 0.2), (8, 1024, 9, 0.3)])
def test_open_loop_rule_one_reevaluated(d, K, period, alpha):
    cfg = dict(B=12, K=K, d=d, lam=1.0, alpha0=alpha, sched=0, prune=1, period=period, sticky=0)
    T = 160 if K < 1024 else 90
    say(f"[nonsticky] open loop d={d} K={K} period={period} T={T}")
    X, R = random_contexts(500 + d + K, T, cfg["B"], d)
    a, m, s, tuner, rec = run_open_loop(cfg, X, R)
    st = parity.compare_open_loop(f"nonsticky d={d} K={K}", cfg, X, R, a, m, s, g_gap=rec["gap"])
    compare_model(tuner, st["oracle"], range(cfg["B"]), 1e-3, 1e-4)
    back = _returns(m, K)
    say(f"[nonsticky] d={d} K={K}: arms back {back}, max score err {st['max_score_err']:.2e}, "
        f"forced {st['forced']}/{st['decisions']}, prune forced {st['forced_prune']}")
    assert back > 0, "no removed arm came back"


def test_open_loop_with_refinement_and_switch():
    cfg = dict(B=10, K=120, d=16, lam=1.0, alpha0=0.3, sched=0, prune=1, period=6, sticky=0,
               refine=dict(refine_period=10, refine_stride=8, refine_half=6, refine_mature=40,
                           refine_min_n=2),
               exploit=dict(ph_delta=0.05, ph_lambda=5.0, ph_window=40, ph_min_rounds=60))
    X, R = random_contexts(77, 200, cfg["B"], cfg["d"])
    R[100:, ::2] -= 1.5
    a, m, s, tuner, rec = run_open_loop(cfg, X, R)
    st = parity.compare_open_loop("nonsticky + refine + switch", cfg, X, R, a, m, s, g_ph=rec["ph"],
                                  g_win=rec["win"], g_gap=rec["gap"])
    say(f"[nonsticky] refine+switch: arms back {_returns(m, cfg['K'])}, refinements "
        f"{st['refinements']}, greedy {st['greedy_decisions']}/{st['decisions']}, "
        f"max score err {st['max_score_err']:.2e}, forced {st['forced']}")
    assert st["refinements"] > 0 and st["greedy_decisions"] > 0


def _closed(wl, probes):
    say(f"[nonsticky] {wl.name} B={wl.B} K={wl.K} d={wl.d} T={wl.T} probes={len(probes)}")
    arr, noi = exogenous(wl)
    out = run_closed_loop(wl, ENV, arr, noi, probes=probes, scores=True)
    st = parity.compare(wl, wl.T, probes, out["probes"])
    wth, wai = compare_model(out["tuner"], st["oracle"], probes, 1e-3, 1e-4)
    back = _returns(out["probes"]["mask"].numpy(), wl.K)
    say(f"[nonsticky] {wl.name}: arms back {back}, max score err {st['max_score_err']:.2e}, "
        f"ctx err {st['max_ctx_err']:.2e}, forced {st['forced']}/{st['decisions']}, prune forced "
        f"{st['forced_prune']}, theta err {wth:.2e}, Ainv err {wai:.2e}")
    return st, back


@pytest.mark.parametrize("name,kw", [("cfg3n", dict(B=16, T=300)), ("cfg4n", dict(B=24, T=300)),
                                     ("cfg5n", dict(B=8, T=300))])
def test_small_closed_loop(name, kw):
    wl = get_workload(name, **kw)
    _closed(wl, list(range(wl.B)))


@pytest.mark.parametrize("name", ["cfg3n", "cfg4n", "cfg5n"])
def test_full_size_closed_loop(name):
    wl = get_workload(name)
    _closed(wl, probe_instances(wl.B, 64))
    torch.cuda.empty_cache()
