"""bench.py end to end on the GPU: one short run and the fields of its JSON
line (the contract the benchmark driver reads)."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_json_line():
    cmd = [sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--workload", "cfg2", "--steps", "30",
           "--warmup", "3", "--cpu-budget", "1"]
    print("[bench test]", " ".join(cmd[2:]), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=280, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert len(lines) == 1, r.stdout
    d = json.loads(lines[0])
    assert d["metric"].startswith("bandit decision-steps/sec")
    assert d["unit"] == "decision-steps/s" and d["value"] > 0
    assert d["n_gpus"] == 1 and d["steps"] == 30 and d["warmup"] == 3
    assert d["higher_is_better"] is True and d["scaling"] == "weak" and d["vs_baseline"] is None
    assert d["dtype"] == "f32" and d["data"].startswith("synthetic")
    assert d["config"]["workload"].startswith("cfg2")
    # throughput is B * steps over the timed region
    assert abs(d["value"] - 4096 * 30 / (d["ms_per_step"] * 30 * 1e-3)) < 1e-6 * d["value"]
    rf = d["roofline"]
    assert rf["bound"] == "hbm" and rf["unit"] == "GB/s" and rf["peak"] == 8000.0
    assert rf["achieved"] > 0 and abs(rf["frac"] - rf["achieved"] / rf["peak"]) < 1e-12
    # the committed counters were taken on cfg4, so none are reported here
    assert rf["traffic"] is None
    det = d["detail"]
    assert 0 < det["step_kernel_avg_ms"] < d["ms_per_step"]
    assert abs(rf["achieved"] - det["algorithmic_bytes_per_launch"] / (det["step_kernel_avg_ms"] * 1e-3) / 1e9) \
        < 1e-6 * rf["achieved"]
    cb = d["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["unit"] == "decision-steps/s" and cb["value"] > 0
    assert cb["cores"] >= 1 and "cfg2" in cb["sample"]
    assert det["cpu_oracle_1thread"]["cores"] == 1
    assert det["host_cpu"]["cpus_visible"] >= 1 and "model" in det["host_cpu"]
    # cfg2: one-wavefront workgroups, packed tails (nothing prunes its arms),
    # no cap on workgroups per compute unit
    assert det["launch_shape"] == {"waves": 1, "simd_waves": 7, "tail_floats": 3, "early_update": 1,
                                   "cu_workgroups": 0}
    assert rf["byte_model"]["model_bytes_per_arm"] == 176 and rf["byte_model"]["dense_bytes_per_arm"] == 288
    # the stream ceiling on cfg2's layout: reading alone is faster than
    # reading plus the write-back, and the step kernel reaches neither
    ce = rf["ceiling"]
    assert ce["read_gbs"] > 0 and ce["read_writeback_gbs"] > 0
    assert abs(ce["achieved_over_read_writeback"] - rf["achieved"] / ce["read_writeback_gbs"]) < 1e-9
    assert 0 < ce["achieved_over_read_writeback"] < 1.2 and "cfg2" in ce["what"]
    for when in ("after_headline", "after_idle"):
        assert 0 < ce[when]["read_writeback_gbs"] <= ce["read_writeback_gbs"]
        assert 0 < ce[when]["read_gbs"] <= ce["read_gbs"]
        # every cap the device admits was timed, the fastest kept
        by_cap = ce[when]["by_cap"]
        assert "0" in by_cap and set(by_cap) <= {"0", "6", "5", "4", "3"}
        assert by_cap[str(ce[when]["read_writeback_cap"])]["read_writeback_us"] == \
            min(v["read_writeback_us"] for v in by_cap.values())
    # every workload over its whole horizon beside the headline
    wls = det["workloads"]
    assert set(wls) == {"cfg1", "cfg2", "cfg3", "cfg4", "cfg5"}
    for name, w in wls.items():
        steps = {"cfg1": 10000, "cfg2": 2000, "cfg3": 1000, "cfg4": 500, "cfg5": 2000}[name]
        assert w["steps"] == steps and w["decision_steps_per_s"] > 0 and 0 < w["frac"] < 1.5
        assert 0 < w["step_kernel_avg_ms"] < w["ms_per_step"] and w["mean_scored_arms"] > 0
        # the stream ceiling on each workload's layout (the headline's own for
        # cfg2), none for the single instance of cfg1
        if name == "cfg1":
            assert w["ceiling_read_writeback_gbs"] is None and w["of_ceiling"] is None
        else:
            assert w["ceiling_read_writeback_gbs"] > 0
            assert abs(w["of_ceiling"] - w["achieved_gbs"] / w["ceiling_read_writeback_gbs"]) < 1e-9
            assert 0 < w["of_ceiling"] < 1.2
    assert wls["cfg2"]["ceiling_read_writeback_gbs"] == ce["read_writeback_gbs"]
