"""How the step kernel is launched for every workload and variant (CPU:
agft_launch_shape_for does no device work).  The table pins the host rules
that choose the record layout, the workgroup width, the register target,
where the update runs and the cap on workgroups per compute unit, each
measured on MI355X (the measurements sit beside the rules in the kernel
source)."""
import pytest

import paper_2508_01744_amd._lib as L
from agft_workloads import get_workload
from paper_2508_01744_amd import launch_shape, make_config, workload_config

# workload: (wavefronts per workgroup, wavefronts per SIMD, tail floats, early
# update, workgroups per compute unit)
EXPECTED = {
    "cfg1": (1, 7, 4, 1, 0), "cfg2": (1, 7, 3, 1, 0), "cfg3": (4, 6, 3, 1, 4), "cfg4": (4, 6, 3, 1, 4),
    "cfg5": (4, 4, 3, 0, 0),
    "cfg2p": (1, 7, 4, 1, 0), "cfg3p": (4, 7, 3, 1, 0), "cfg4p": (4, 7, 3, 1, 0), "cfg5p": (4, 4, 3, 0, 0),
    "cfg1e": (1, 7, 4, 1, 0), "cfg2e": (1, 7, 4, 1, 0), "cfg3e": (1, 6, 3, 1, 0), "cfg4e": (1, 6, 3, 1, 0),
    "cfg5e": (4, 4, 3, 0, 0), "cfg4pe": (1, 7, 3, 1, 0),
    "cfg2r": (1, 7, 4, 1, 0), "cfg3r": (1, 7, 4, 1, 0), "cfg4r": (1, 7, 4, 1, 0), "cfg5r": (4, 4, 3, 0, 0),
    "cfg4per": (1, 7, 4, 1, 0), "cfg3n": (4, 6, 3, 1, 4), "cfg4n": (4, 6, 3, 1, 4), "cfg5n": (4, 4, 3, 0, 0),
}


@pytest.mark.parametrize("name", sorted(EXPECTED))
def test_workload_launch_shapes(name):
    s = launch_shape(workload_config(get_workload(name)))
    assert (s["waves"], s["simd_waves"], s["tail_floats"], s["early_update"], s["cu_workgroups"]) == EXPECTED[name]


def test_rules_at_their_thresholds():
    def shape(**kw):
        base = dict(B=64, K=128, d=16, alpha0=0.5, prune_rule=1, prune_period=50)
        base.update(kw)
        return launch_shape(make_config(**base))
    # 16 KB of records per exploring instance: 26 arms of 608 bytes at d = 16
    assert shape(K=26)["tail_floats"] == 4 and shape(K=27)["tail_floats"] == 3
    # 8 KB where nothing prunes or restricts the arms: 13 and 14 arms at d = 16
    assert shape(K=13, prune_rule=0)["tail_floats"] == 4 and shape(K=14, prune_rule=0)["tail_floats"] == 3
    assert shape(K=14)["tail_floats"] == 4
    assert shape(K=26)["waves"] == 1 and shape(K=27)["waves"] == 4
    # the paper's rules keep seven wavefronts per SIMD at d = 16
    rules = dict(ext_rounds=60, ext_min_n=3, ext_thr=-1.2, hist_after=30, hist_min_n=6, hist_kappa=1.0,
                 hist_min_arms=3, cascade_k=48)
    assert shape()["simd_waves"] == 6 and shape(prune_rule=15, heuristics=rules)["simd_waves"] == 7
    # four workgroups per compute unit only for four-wavefront workgroups at six per SIMD
    assert shape()["cu_workgroups"] == 4 and shape(prune_rule=15, heuristics=rules)["cu_workgroups"] == 0
    assert shape(K=26)["cu_workgroups"] == 0 and shape(d=32)["cu_workgroups"] == 0
    # d = 32 updates after the stream only when it streams more than 16 KB
    assert shape(d=32, K=7)["early_update"] == 1 and shape(d=32, K=8)["early_update"] == 0
    assert shape(d=8, K=1024)["early_update"] == 1


def test_invalid_configuration():
    code, _ = L.agft_launch_shape_for(make_config(0, 16, 8))
    assert code == L.AGFT_E_INVAL
