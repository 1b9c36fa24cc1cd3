"""GPU step vs the fp64 oracle on the five workloads (closed loop).

Small cases record every instance at every step; full-size cases run the
whole batch at the benchmark's launch configuration and record 64 probe
instances (strided, first and last) at every step."""
import pytest
import torch

import parity
from agft_workloads import ENV, exogenous, get_workload, probe_instances
from gpu_helpers import compare_model, say
from paper_2508_01744_amd import run_closed_loop

pytestmark = pytest.mark.gpu

SMALL = {1: dict(T=3000), 2: dict(B=48, T=400), 3: dict(B=24, T=300),
         4: dict(B=40, T=300), 5: dict(B=12, T=300)}

# theta and A^{-1} after the run, relative to max(1, max |entry|)
THETA_TOL, AINV_TOL = 1e-3, 1e-4


def _run_and_compare(wl, probes):
    say(f"[parity] {wl.name} B={wl.B} K={wl.K} d={wl.d} T={wl.T} probes={len(probes)}")
    arr, noi = exogenous(wl)
    out = run_closed_loop(wl, ENV, arr, noi, probes=probes, scores=True)
    st = parity.compare(wl, wl.T, probes, out["probes"])
    wth, wai = compare_model(out["tuner"], st["oracle"], probes, THETA_TOL, AINV_TOL)
    say(f"[parity] {wl.name}: max score err {st['max_score_err']:.2e} (relative, |s| >= 1: "
        f"{st['max_rel_err_abs_ge_1']:.2e}; absolute, |s| < 1: {st['max_abs_err_abs_lt_1']:.2e}), ctx err "
        f"{st['max_ctx_err']:.2e}, reward err {st['max_reward_err']:.2e}, forced "
        f"{st['forced']}/{st['decisions']}, prune forced {st['forced_prune']}, rules forced "
        f"{st['forced_rules']}, exact-tie steps "
        f"{st['exact_tie_steps']}, gap err {st['max_gap_err']:.2e}, theta err {wth:.2e}, "
        f"Ainv err {wai:.2e}")
    return st


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_small_every_instance(cfg):
    wl = get_workload(cfg, **SMALL[cfg])
    _run_and_compare(wl, list(range(wl.B)))


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_full_size_probes(cfg):
    wl = get_workload(cfg)
    _run_and_compare(wl, probe_instances(wl.B, 64))
    torch.cuda.empty_cache()


@pytest.mark.parametrize("cfg", ["cfg2p", "cfg3p", "cfg4p", "cfg5p"])
def test_small_paper_pruning(cfg):
    """The workloads with the paper's pruning rules added (Sec. 4.3)."""
    small = {"cfg2p": dict(B=32, T=400), "cfg3p": dict(B=16, T=300), "cfg4p": dict(B=24, T=300),
             "cfg5p": dict(B=8, T=300)}
    wl = get_workload(cfg, **small[cfg])
    _run_and_compare(wl, list(range(wl.B)))


@pytest.mark.parametrize("cfg", ["cfg2p", "cfg3p", "cfg4p", "cfg5p"])
def test_full_size_paper_pruning(cfg):
    wl = get_workload(cfg)
    _run_and_compare(wl, probe_instances(wl.B, 64))
    torch.cuda.empty_cache()


def test_ragged_arms_closed_loop():
    """K = 100 arms (two wavefronts, the second 28 lanes short), pruning."""
    wl = get_workload(3, B=20, K=100, T=250)
    _run_and_compare(wl, list(range(wl.B)))
