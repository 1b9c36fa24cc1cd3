"""Mixed-maturity refinement of the action space (Sec. 4.4) on the GPU
against the oracle: the coarse starting grid, the statistical and predictive
anchors, the 2h+1-arm windows, and their interplay with the pruning rules and
the switch to exploitation.

Open loop (the same contexts and rewards to both sides) with short refinement
periods so that windows move often; closed loop on the workloads with the
refinement enabled."""
import pytest
import torch

import parity
from agft_workloads import ENV, exogenous, get_workload, probe_instances
from gpu_helpers import compare_model, random_contexts, run_open_loop, say
from paper_2508_01744_amd import GpuEnv, Tuner, env_config, run_closed_loop

pytestmark = pytest.mark.gpu

FAST_REFINE = dict(refine_period=7, refine_stride=5, refine_half=3, refine_mature=30,
                   refine_min_n=2)


def _open_loop(name, cfg, T, seed):
    say(f"[refine] {name}: {cfg} T={T}")
    X, R = random_contexts(seed, T, cfg["B"], cfg["d"])
    a, m, s, tuner, rec = run_open_loop(cfg, X, R)
    st = parity.compare_open_loop(name, cfg, X, R, a, m, s, g_ph=rec["ph"], g_win=rec["win"])
    compare_model(tuner, st["oracle"], range(cfg["B"]), 1e-3, 1e-4)
    say(f"[refine] {name}: refinements {st['refinements']}, windows forced {st['forced_window']}, "
        f"max score err {st['max_score_err']:.2e}, forced {st['forced']}/{st['decisions']}")
    assert st["refinements"] > 0
    return st, rec


@pytest.mark.parametrize("d,K,prune,period", [(8, 40, 0, 50), (16, 128, 1, 11), (32, 33, 1, 9),
                                              (16, 100, 1, 13), (8, 1024, 1, 20)])
def test_open_loop_refinement(d, K, prune, period):
    cfg = dict(B=12, K=K, d=d, lam=1.0, alpha0=0.5, sched=0, prune=prune, period=period,
               heuristics=None, refine=FAST_REFINE)
    T = 90 if K < 1024 else 60
    _open_loop(f"refine d={d} K={K}", cfg, T, 500 + d + K)


def test_open_loop_refinement_with_rules_and_switch():
    """Every option at once: rules 1-8, the switch and the refinement."""
    cfg = dict(B=12, K=60, d=16, lam=1.0, alpha0=0.6, sched=0, prune=15, period=25,
               heuristics=dict(ext_rounds=40, ext_min_n=1, ext_thr=-1.0, hist_after=10,
                               hist_min_n=2, hist_kappa=0.5, hist_min_arms=3, cascade_k=30),
               exploit=dict(ph_delta=0.05, ph_lambda=5.0, ph_window=40, ph_min_rounds=60),
               refine=FAST_REFINE)
    st, rec = _open_loop("refine + rules 15 + switch", cfg, 160, 88)
    assert st["greedy_decisions"] > 0


def test_window_of_one_arm():
    """refine_half = 0: after the first refinement only the anchor is in play."""
    cfg = dict(B=6, K=24, d=8, lam=1.0, alpha0=0.5, sched=0, prune=0, period=50, heuristics=None,
               refine=dict(FAST_REFINE, refine_half=0))
    st, rec = _open_loop("refine half=0", cfg, 40, 3)
    w = rec["win"][-1]
    assert (w[:, 0] == w[:, 1]).all()


SMALL = {"cfg2r": dict(B=32, T=400), "cfg3r": dict(B=16, T=300), "cfg4r": dict(B=24, T=300),
         "cfg5r": dict(B=8, T=300), "cfg4per": dict(B=24, T=300)}


def _closed(wl, probes):
    say(f"[refine] {wl.name} B={wl.B} K={wl.K} d={wl.d} T={wl.T} probes={len(probes)}")
    arr, noi = exogenous(wl)
    out = run_closed_loop(wl, ENV, arr, noi, probes=probes, scores=True)
    st = parity.compare(wl, wl.T, probes, out["probes"])
    wth, wai = compare_model(out["tuner"], st["oracle"], probes, 1e-3, 1e-4)
    say(f"[refine] {wl.name}: refinements {st['refinements']}, windows forced {st['forced_window']}, "
        f"max score err {st['max_score_err']:.2e}, forced {st['forced']}/{st['decisions']}, "
        f"theta err {wth:.2e}, Ainv err {wai:.2e}")
    assert st["refinements"] > 0
    return st


@pytest.mark.parametrize("name", list(SMALL))
def test_small_closed_loop(name):
    wl = get_workload(name, **SMALL[name])
    _closed(wl, list(range(wl.B)))


@pytest.mark.parametrize("name", ["cfg2r", "cfg3r", "cfg4r", "cfg5r", "cfg4per"])
def test_full_size_closed_loop(name):
    wl = get_workload(name)
    _closed(wl, probe_instances(wl.B, 64))
    torch.cuda.empty_cache()


def test_resume_with_refinement_is_bit_identical():
    """Save the buffer after some refinements, adopt it, go on."""
    wl = get_workload("cfg3r", B=16, T=220)
    arr, noi = exogenous(wl)
    dev = torch.device("cuda")
    full = run_closed_loop(wl, ENV, arr, noi, probes=range(wl.B))
    T1 = 133
    env = GpuEnv(env_config(wl, ENV), torch.as_tensor(arr, device=dev), torch.as_tensor(noi, device=dev))
    tun = Tuner.from_workload(wl, device=dev)
    act = torch.empty(wl.B, dtype=torch.int32, device=dev)
    x, r, acts = env.reset(), None, []
    for t in range(wl.T):
        if t == T1:
            assert (tun.view()["window"][:, 2] == 1).any()
            saved = tun.state.clone()
            tun.close()
            tun = Tuner.from_workload(wl, device=dev, state=saved, adopt=True)
        tun.step(x, r, act)
        acts.append(act.clone())
        r, x = env.step(t, act)
    tun.flush(r)
    torch.cuda.synchronize()
    assert torch.equal(torch.stack(acts).cpu(), full["probes"]["a"])
    assert torch.equal(tun.state, full["tuner"].state)
