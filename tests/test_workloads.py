"""Seeded input generators (CPU only)."""
import numpy as np

from agft_workloads import WORKLOADS, exogenous, get_workload, probe_instances, arm_values


def test_configs_match_their_descriptions():
    sizes = {c: (w.B, w.K, w.d, w.T) for c, w in WORKLOADS.items()}
    assert sizes == {1: (1, 16, 8, 10_000), 2: (4096, 64, 8, 2000), 3: (16_384, 128, 16, 1000),
                     4: (65_536, 128, 16, 500), 5: (1024, 256, 32, 2000)}
    assert [WORKLOADS[c].prune for c in range(1, 6)] == [0, 0, 1, 1, 1]
    assert WORKLOADS[5].alpha_sched == 1 and WORKLOADS[5].drift == 0.3
    assert abs(WORKLOADS[5].alpha_at(3) - 0.5) < 1e-15


def test_subset_regeneration_matches_full_batch():
    wl = get_workload(2, B=64, T=50)
    a, n = exogenous(wl)
    idx = [0, 7, 63]
    a2, n2 = exogenous(wl, idx)
    assert np.array_equal(a[:, idx], a2) and np.array_equal(n[:, idx], n2)
    a3, n3 = exogenous(wl)
    assert np.array_equal(a, a3) and np.array_equal(n, n3)


def test_trace_statistics():
    wl = get_workload(4, B=256, T=500)
    a, n = exogenous(wl)
    assert a.shape == (501, 256) and a.dtype == np.int32 and n.dtype == np.float32
    assert 0.015 < n.std() < 0.025
    # on/off traces: per-instance arrival means sit between the off and on rates
    m = a.mean(axis=0)
    assert m.min() > 0.3 and m.max() < 21
    wl = get_workload(2, B=256, T=2000)
    a, _ = exogenous(wl)
    m = a.mean(axis=0)
    assert 0.1 < m.min() and m.max() < 22


def test_probe_instances_and_arms():
    p = probe_instances(65_536)
    assert p[0] == 0 and p[-1] == 65_535 and len(p) == 64
    assert probe_instances(10) == list(range(10))
    v = arm_values(128)
    assert v[0] == 0.2 and abs(v[-1] - 1.0) < 1e-15 and len(v) == 128
