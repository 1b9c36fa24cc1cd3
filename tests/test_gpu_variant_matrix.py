"""Every workload family with every combination of the options that the
dedicated tests do not already run closed loop: the paper's rules (p), the
switch to exploitation (e) and the refinement (r), on small batches, each
side with its own environment on the same draws.  Every context, reward,
score, prune bit, action, test state and action space is compared at every
step, and the final models through the export kernel."""
import pytest

import parity
from agft_workloads import ENV, exogenous, get_workload
from gpu_helpers import compare_model, say
from paper_2508_01744_amd import run_closed_loop

pytestmark = pytest.mark.gpu

COVERED = {"cfg2p", "cfg3p", "cfg4p", "cfg5p", "cfg2e", "cfg3e", "cfg4e", "cfg5e", "cfg4pe",
           "cfg2r", "cfg3r", "cfg4r", "cfg5r", "cfg4per"}
CASES = [f"cfg{c}{s}" for c in range(1, 6) for s in ("p", "e", "r", "pe", "pr", "er", "per")
         if f"cfg{c}{s}" not in COVERED]


@pytest.mark.parametrize("name", CASES)
def test_variant_closed_loop(name):
    wl = get_workload(name, B=6, T=260)
    say(f"[matrix] {wl.name} B={wl.B} K={wl.K} d={wl.d} T={wl.T}")
    arr, noi = exogenous(wl)
    out = run_closed_loop(wl, ENV, arr, noi, probes=list(range(wl.B)), scores=True)
    st = parity.compare(wl, wl.T, list(range(wl.B)), out["probes"])
    compare_model(out["tuner"], st["oracle"], list(range(wl.B)), 1e-3, 1e-4)
    say(f"[matrix] {wl.name}: max score err {st['max_score_err']:.2e}, forced {st['forced']}/{st['decisions']}, "
        f"greedy {st.get('greedy_decisions', 0)}, refinements {st.get('refinements', 0)}")
