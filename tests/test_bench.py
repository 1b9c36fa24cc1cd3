"""bench.py's contract on the CPU: the one-GPU guard, the algorithmic byte
count the roofline divides by, the rule that measured traffic is reported
only for the kernel source and workload it was taken on, and the fields of
the oracle baselines, and that the stream ceiling's failure is reported, not
fatal."""
import json
import os
import subprocess
import sys

import pytest

import bench
from agft_workloads import get_workload

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_step_bytes_worked_cases():
    # cfg4: d = 16, 152 floats of model per arm, 4 mask words per instance
    wl = get_workload("cfg4")
    B = wl.B
    per_inst = (4 * 152 * (127 + 2)     # 127 other arms read, the updated arm read and written
                + 4 * (3 * 16 + 7)      # context, stashed context, words
                + 4 * 4)                # mask words read
    assert bench.step_bytes(wl, 127 * B, 0, False, True) == B * per_inst
    # the first step has no update; a pruning step writes the mask back
    assert bench.step_bytes(wl, 128 * B, 0, True, False) == B * (4 * 152 * 128 + 4 * 55 + 32)
    # an exploiting instance reads theta alone: 64 bytes per arm at d = 16
    assert (bench.step_bytes(wl, 0, 127 * B, False, True) - bench.step_bytes(wl, 0, 0, False, True)
            == B * 127 * 64)
    # the paper's rules add the per-arm statistics (read by the rules, and the
    # updated arm's count and sum kept); the switch its test words
    wp, we = get_workload("cfg4p"), get_workload("cfg4e")
    base = bench.step_bytes(wl, 0, 0, False, True)
    assert bench.step_bytes(wp, 0, 0, False, True) - base == B * (8 * 128 + 16)
    assert bench.step_bytes(we, 0, 0, False, True) - base == B * 72


def test_traffic_only_for_the_profiled_source_and_workload(tmp_path):
    src = tmp_path / "kernel.hip"
    src.write_text("kernel source\n")
    path = tmp_path / "counters.json"

    def write(**kw):
        rec = dict(workload="cfg4", source_sha256_16=bench.source_hash(str(src)), hbm_bytes_per_launch=5.1e9)
        rec.update(kw)
        path.write_text(json.dumps(rec))

    write()
    assert bench.counter_traffic("cfg4", str(path), str(src)) == 5.1e9
    assert bench.counter_traffic("cfg3", str(path), str(src)) is None
    # counters taken over another window of steps are not this run's traffic
    write(steps=20, warmup=5)
    assert bench.counter_traffic("cfg4", str(path), str(src), steps=20, warmup=5) == 5.1e9
    assert bench.counter_traffic("cfg4", str(path), str(src), steps=500, warmup=5) is None
    assert bench.counter_traffic("cfg4", str(path), str(src), steps=20, warmup=20) is None
    # per-step counters of a fresh run serve any window within them: the mean
    # of its first `steps` steps, whatever the warm-up
    write(per_step_hbm_bytes=[5.0e9, 5.2e9, 5.4e9, 5.6e9])
    assert bench.counter_traffic("cfg4", str(path), str(src), steps=2, warmup=5) == 5.1e9
    assert abs(bench.counter_traffic("cfg4", str(path), str(src), steps=4, warmup=20) - 5.3e9) < 1.0
    assert bench.counter_traffic("cfg4", str(path), str(src), steps=5, warmup=5) is None
    assert bench.counter_traffic("cfg4", str(path), str(src)) is None
    write()
    src.write_text("kernel source, changed\n")
    assert bench.counter_traffic("cfg4", str(path), str(src)) is None
    assert bench.counter_traffic("cfg4", str(tmp_path / "absent.json"), str(src)) is None


def test_oracle_baselines():
    wl = get_workload("cfg2", B=64, T=30)
    allc = bench.cpu_baseline(wl, 5.0)
    assert allc["kind"] == "oracle" and allc["unit"] == "decision-steps/s" and allc["value"] > 0
    assert allc["cores"] >= 1 and allc["n"] == 64 and allc["steps"] == 30
    one = bench.cpu_baseline(wl, 5.0, threads=1, max_steps=10, n_max=8)
    assert one["cores"] == 1 and one["n"] == 8 and one["steps"] == 10
    # the thread count is restored afterwards
    assert bench.cpu_baseline(wl, 5.0, max_steps=1)["cores"] == allc["cores"]


def test_byte_model_states_both_layouts():
    bm = bench.byte_model(get_workload("cfg4"))
    assert bm["model_bytes_per_arm"] == 608 and bm["dense_bytes_per_arm"] == 1088
    bm = bench.byte_model(get_workload("cfg5"))
    assert bm["model_bytes_per_arm"] == 4 * (32 + 528) and bm["dense_bytes_per_arm"] == 4 * (1024 + 32)


def test_ceiling_failure_does_not_sink_the_line(monkeypatch):
    """The stream ceiling is a side measurement: if its library cannot run,
    stream_ceiling raises a RuntimeError that main() records in the line."""
    monkeypatch.setattr(bench, "CEILING_LIB", "/nonexistent/libagft_ceiling.so")
    wl = get_workload("cfg2")
    with pytest.raises(RuntimeError, match="not built"):
        bench.stream_ceiling(wl)


def test_host_cpu_is_described():
    h = bench.host_cpu()
    assert h["cpus_visible"] >= 1 and h["cpus_machine"] >= h["cpus_visible"]
    assert h["model"] is None or isinstance(h["model"], str)
