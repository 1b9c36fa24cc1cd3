"""Benchmark of the batched AGFT decide-and-update step on one MI355X.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload cfg4]

A step is one decision for every instance of the workload: the tuner step
kernel (pending update, scoring of every active arm, pruning, argmax) and the
environment kernel that produces the next contexts and rewards.  All inputs
(state, exogenous draws) are resident in HBM before the timed region, which
times exactly K steps from a freshly initialised state.  Then each of the five
workloads is timed the same way over its whole horizon (detail.workloads).
Prints one JSON line.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0   # MI355X HBM3E, AMD's published peak
STEP_SRC = os.path.join(ROOT, "paper_2508_01744_amd", "csrc", "agft_step.hip")
COUNTERS = os.path.join(ROOT, "profiles", "agft_step_counters.json")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def source_hash(path=STEP_SRC):
    with open(path, "rb") as fh:
        return hashlib.sha256(fh.read()).hexdigest()[:16]


class TimingEvent:
    """A HIP event for timing only, recorded on a torch stream: created with
    hipEventDisableSystemFence, so that recording it does not write back and
    invalidate the caches the way a default event does (that costs about
    3 us per record and lands on the launch being timed)."""
    _hip = None
    FLAGS = 0x20000000   # hipEventDisableSystemFence

    @classmethod
    def _lib(cls):
        if cls._hip is None:
            import ctypes
            from paper_2508_01744_amd import _lib
            # the HIP runtime the step kernel's library is bound to (symbol
            # lookup through its handle reaches its dependencies)
            lib = ctypes.CDLL(_lib.LIB_PATH)
            vp = ctypes.c_void_p
            lib.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(vp), ctypes.c_uint]
            lib.hipEventRecord.argtypes = [vp, vp]
            lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), vp, vp]
            lib.hipEventDestroy.argtypes = [vp]
            for f in (lib.hipEventCreateWithFlags, lib.hipEventRecord, lib.hipEventElapsedTime,
                      lib.hipEventDestroy):
                f.restype = ctypes.c_int
            cls._hip = lib
        return cls._hip

    def __init__(self):
        import ctypes
        self._ev = ctypes.c_void_p()
        rc = self._lib().hipEventCreateWithFlags(ctypes.byref(self._ev), self.FLAGS)
        if rc != 0:
            raise RuntimeError(f"hipEventCreateWithFlags failed ({rc})")

    def record(self, stream):
        rc = self._lib().hipEventRecord(self._ev, stream.cuda_stream)
        if rc != 0:
            raise RuntimeError(f"hipEventRecord failed ({rc})")

    def elapsed_time(self, end):
        import ctypes
        ms = ctypes.c_float()
        rc = self._lib().hipEventElapsedTime(ctypes.byref(ms), self._ev, end._ev)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return ms.value

    def __del__(self):
        if self._hip is not None and getattr(self, "_ev", None):
            self._hip.hipEventDestroy(self._ev)


def counter_traffic(workload, path=COUNTERS, source=STEP_SRC, steps=None, warmup=None):
    """HBM bytes per step-kernel launch from the committed counter summary,
    or None unless it was taken on this workload with this kernel source.

    The summary holds the bytes of every step of a fresh run
    (per_step_hbm_bytes[t], t = 0, 1, ...): a bench run times its steps from
    a fresh state on the same draws, so its window is the first `steps` of
    them, whatever its warm-up (None if the summary covers fewer steps).  A
    summary with one figure for a window (steps, warmup) serves only that
    window."""
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        cnt = json.load(fh)
    if cnt.get("source_sha256_16") != source_hash(source) or cnt.get("workload") != workload:
        return None
    per_step = cnt.get("per_step_hbm_bytes")
    if per_step is not None:
        if steps is None:
            return None
        return sum(per_step[:steps]) / steps if 0 < steps <= len(per_step) else None
    if steps is not None and (cnt.get("steps"), cnt.get("warmup")) != (steps, warmup):
        return None
    return cnt.get("hbm_bytes_per_launch")


def record_floats(d):
    return d + d * (d + 1) // 2


def step_bytes(wl, scored_exploring, scored_greedy, mask_write, update):
    """Algorithmic HBM bytes of one step kernel launch.

    Per instance: the previous decision's arm is read and written back once
    (its model: the d(d+1)/2 factor entries and theta, with its reward count
    and sum when a rule reads those); every other arm scored is read once, as its whole model while
    the instance explores (Eq. 1) and as theta alone once it exploits (Eq. 2);
    plus context, stashed context, reward, action and bookkeeping words, the
    per-arm reward statistics when the paper's rules 2-8 are on, the
    Page-Hinkley words when the switch is on, and the action-set mask (written
    back when a rule may remove arms).  scored_*: arms scored, the previous
    decision's arm excluded, summed over the instances in each mode.
    """
    B, d = wl.B, wl.d
    s = record_floats(d)
    kw = (wl.K + 31) // 32
    upd = B if update else 0
    stats_kept = bool(wl.prune & 14) or bool(wl.refine)
    records = 4 * s * (scored_exploring + 2 * upd) + 4 * d * scored_greedy + (16 * upd if stats_kept else 0)
    io = B * 4 * (3 * d + 7)           # ctx, xprev r/w; reward, action, aprev r/w, kact, bad
    if wl.prune & 14:
        io += B * 8 * wl.K             # per-arm count and reward sum
    if wl.exploit:
        io += B * 4 * 9 * 2            # mode and test state r/w
    mask = B * 4 * kw * (2 if mask_write else 1)
    return float(records + io + mask)


def cpu_baseline(wl, budget_s, threads=None, n_max=16384, max_steps=None):
    """The fp64 oracle (C, OpenMP over instances) with its fp64 environment,
    closed loop, on a bounded sample of the workload's instances and steps
    (threads: the OpenMP thread count, default all)."""
    from agft_workloads import exogenous
    from oracle import Env, Oracle
    n = min(wl.B, n_max)
    all_threads = Oracle.threads()
    if threads is not None:
        Oracle.set_threads(threads)
    T = wl.T
    arr, noi = exogenous(wl, range(n), T)
    env = Env(wl, arr, noi, T)
    ora = Oracle.from_workload(wl, B=n)
    x = env.reset()
    r = None
    t0 = time.perf_counter()
    steps = 0
    for t in range(T if max_steps is None else min(T, max_steps)):
        ucb, lcb, keep, action = ora.decide(x, r)
        ora.commit(x, action, keep)
        r, x = env.step(t, action)
        steps += 1
        if time.perf_counter() - t0 > budget_s:
            break
    el = time.perf_counter() - t0
    cores = Oracle.threads()
    Oracle.set_threads(all_threads)
    return dict(value=n * steps / el, unit="decision-steps/s", cores=cores, kind="oracle",
                sample=f"{n} instances x {steps} steps of {wl.name} (closed loop with the fp64 "
                       f"environment, {el:.1f} s)", n=n, steps=steps)


def host_cpu():
    """The host processor the oracle baseline ran on: model name, logical
    CPUs visible to this process and in the machine."""
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    visible = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    return {"model": model, "cpus_visible": visible, "cpus_machine": os.cpu_count()}


def measure(wl, K, W, dev, log_prefix="[bench]", draws=None):
    """Run W untimed warm-up steps of workload wl, re-initialise, time K steps
    from the fresh state (the step and environment kernels of each step),
    replay them untimed to count the arms each step scored, and return the
    figures of one bench line for this workload.  draws: the exogenous
    arrays (arrivals, noise) of at least max(K, W) + 1 windows, if already made."""
    import numpy as np
    import torch
    from agft_workloads import ENV, exogenous
    from paper_2508_01744_amd import GpuEnv, Tuner, env_config

    T_env = max(K, W, 1)
    log(f"{log_prefix} {wl.name}: B={wl.B} K={wl.K} d={wl.d}; timed steps {K}, warmup {W}")
    arr, noi = exogenous(wl, T=T_env) if draws is None else (draws[0][:T_env + 1], draws[1][:T_env + 1])
    arr_d = torch.as_tensor(arr, device=dev)
    noi_d = torch.as_tensor(noi, device=dev)
    del arr, noi
    env = GpuEnv(env_config(wl, ENV, T=T_env), arr_d, noi_d)
    tuner = Tuner.from_workload(wl, device=dev)
    action = torch.empty(wl.B, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev)

    def fresh():
        nonlocal tuner
        state = tuner.state
        tuner.close()
        tuner = Tuner.from_workload(wl, device=dev, state=state)

    def run(nsteps, kernel_events=None, scored_log=None):
        x = env.reset()
        r = None
        if scored_log is not None:
            sc = torch.empty(wl.B, 2, wl.K, device=dev)
            rows = torch.arange(wl.B, device=dev)
            prev = torch.empty_like(action)
            view = tuner.view()
        for t in range(nsteps):
            if kernel_events is not None:
                kernel_events[t][0].record(stream)
            tuner.step(x, r, action, sc if scored_log is not None else None)
            if kernel_events is not None:
                kernel_events[t][1].record(stream)
            if scored_log is not None:
                # arms scored this step, the one updated from the previous decision excluded,
                # split by the instance's mode (the mode word after the step)
                fin = torch.isfinite(sc[:, 0, :])
                if t > 0:
                    ok = prev >= 0
                    fin[rows[ok], prev[ok].long()] = False
                n = fin.sum(dim=1)
                greedy = view["mode"] >= 0
                scored_log.append(torch.stack([(n * ~greedy).sum(), (n * greedy).sum(),
                                               view["kact"].sum(), greedy.sum()]))
                prev.copy_(action)
            r, x = env.step(t, action)

    # warm-up on a fresh state, then re-initialise
    if W > 0:
        run(W)
    torch.cuda.synchronize()
    fresh()
    torch.cuda.synchronize()

    ev = [(TimingEvent(), TimingEvent()) for _ in range(K)]
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    start.record(stream)
    run(K, kernel_events=ev)
    stop.record(stream)
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    elapsed_ms = start.elapsed_time(stop)
    kernel_ms = np.array([a.elapsed_time(b) for a, b in ev])

    # the same steps through agft_sim_step (the environment in the step
    # kernel's epilogue, one launch per step, up to 8,192 instances; the two
    # kernels above)
    fresh()
    torch.cuda.synchronize()
    f0, f1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    env.reset()
    f0.record(stream)
    for t in range(K):
        env.fused_step(tuner, action)
    f1.record(stream)
    torch.cuda.synchronize()
    fused_ms = f0.elapsed_time(f1)

    # the run is deterministic: replay it untimed to log the arms each step scored
    fresh()
    scored_log = []
    run(K, scored_log=scored_log)
    scored = torch.stack(scored_log).cpu().numpy().astype(np.int64) if scored_log else np.zeros((0, 4))
    torch.cuda.synchronize()
    tuner.close()
    del tuner, env, arr_d, noi_d
    torch.cuda.empty_cache()

    total_bytes = 0.0
    for t in range(K):
        mask_write = bool(wl.prune & 14) or (wl.prune & 1 and t > 0 and t % wl.period == 0)
        total_bytes += step_bytes(wl, int(scored[t, 0]), int(scored[t, 1]), mask_write, update=t > 0)
    bytes_per_launch = total_bytes / K
    kernel_avg_ms = float(kernel_ms.mean())
    achieved = bytes_per_launch / (kernel_avg_ms * 1e-3) / 1e9
    return dict(value=wl.B * K / (elapsed_ms * 1e-3), ms_per_step=elapsed_ms / K, steps=K,
                value_fused=wl.B * K / (fused_ms * 1e-3), ms_per_step_fused=fused_ms / K,
                step_kernel_avg_ms=kernel_avg_ms,
                step_kernel_median_ms=float(np.median(kernel_ms)),
                step_kernel_share=float(kernel_ms.sum() / elapsed_ms),
                algorithmic_bytes_per_launch=bytes_per_launch,
                achieved_gbs=achieved, frac=achieved / HBM_PEAK_GBS,
                mean_scored_arms=float(scored[:, :2].sum(axis=1).mean() / wl.B) if K else None,
                mean_active_arms_after_step=float(scored[:, 2].mean() / wl.B) if K else None,
                exploiting_fraction=float(scored[:, 3].mean() / wl.B) if K else None,
                wall_s=t_wall)


def byte_model(wl):
    """What the algorithmic byte count charges per arm, against the dense
    d x d inverse-plus-vector layout a plain implementation of Eq. 1-5 keeps."""
    d = wl.d
    return {"layout": "packed: theta and the upper-triangular factor S (S S^T = A^-1) of each arm",
            "model_bytes_per_arm": 4 * record_floats(d),
            "dense_bytes_per_arm": 4 * (d * d + d),
            "counted": "every scored arm's model read once (theta alone for an exploiting instance), "
                       "the updated arm read and written, the per-instance words and mask"}


def copy_rate(dev, reps):
    """A plain device copy (1 GiB read, 1 GiB written) as the bandwidth
    cross-check of the peak figure; its counter readings also calibrate the
    HBM counters (--calibrate-copy runs it under the profiler)."""
    import torch
    stream = torch.cuda.current_stream(dev)
    a = torch.empty(1 << 28, dtype=torch.float32, device=dev).normal_()
    b = torch.empty_like(a)
    torch.neg(a, out=b)
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record(stream)
    for _ in range(reps):
        torch.neg(a, out=b)
    c1.record(stream)
    torch.cuda.synchronize()
    gbs = reps * 2 * a.numel() * 4 / (c0.elapsed_time(c1) * 1e-3) / 1e9
    del a, b
    torch.cuda.empty_cache()
    return gbs


CEILING_LIB = os.path.join(ROOT, "paper_2508_01744_amd", "libagft_ceiling.so")


# workgroups per compute unit the stream ceiling is measured at (0: uncapped);
# the rate of concurrent instance streams depends on how many run at once,
# so the ceiling is the best of these
CEILING_CAPS = (0, 6, 5, 4, 3)


def stream_ceiling(wl, launches=20, caps=CEILING_CAPS, rest_s=0.0):
    """The attainable HBM rate of the step's memory traffic without its
    arithmetic (libagft_ceiling.so): one workgroup per instance reads every
    chunk of an instance-sized region of the step kernel's record layout,
    then, in the second form, writes one record back, as the step's update
    does; each form at every cap on workgroups per compute unit in `caps`
    that the device admits (after `rest_s` seconds of idle before each
    cap), the fastest kept.  Returns both rates in GB/s
    (bytes moved over the average launch duration), the durations, the caps
    they came from and every cap's durations."""
    import ctypes
    from paper_2508_01744_amd import launch_shape, workload_config
    if not os.path.exists(CEILING_LIB):
        raise RuntimeError(f"{CEILING_LIB} is not built: run __graft_entry__.build()")
    lib = ctypes.CDLL(CEILING_LIB)
    f = lib.agft_stream_ceiling_at
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                  ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]
    tf = launch_shape(workload_config(wl))["tail_floats"]
    nb = 64 // wl.d
    rec = (wl.d // 2) * (wl.d // 4) + (wl.d // 2) * tf // 4      # 16-byte chunks per arm record
    chunks = -(-wl.K // nb) * nb * rec                           # per instance, blocks of nb arms
    by_cap = {}
    for cap in caps:
        if rest_s > 0:
            time.sleep(rest_s)
        r_us, rw_us = ctypes.c_double(), ctypes.c_double()
        code = f(wl.B, chunks, rec, launches, cap, ctypes.byref(r_us), ctypes.byref(rw_us))
        if code == 3:      # the device's occupancy calculator does not confirm this cap
            continue
        if code != 0:
            raise RuntimeError(f"agft_stream_ceiling_at failed ({code}) at {cap} workgroups per compute unit")
        by_cap[cap] = {"read_us": r_us.value, "read_writeback_us": rw_us.value}
    if not by_cap:
        raise RuntimeError("agft_stream_ceiling_at admitted none of the caps")
    cap_r = min(by_cap, key=lambda c: by_cap[c]["read_us"])
    cap_rw = min(by_cap, key=lambda c: by_cap[c]["read_writeback_us"])
    r_us, rw_us = by_cap[cap_r]["read_us"], by_cap[cap_rw]["read_writeback_us"]
    read_b, write_b = wl.B * chunks * 16, wl.B * rec * 16
    return {"read_gbs": read_b / (r_us * 1e-6) / 1e9,
            "read_writeback_gbs": (read_b + write_b) / (rw_us * 1e-6) / 1e9,
            "read_us": r_us, "read_writeback_us": rw_us, "read_cap": cap_r, "read_writeback_cap": cap_rw,
            "by_cap": {str(c): v for c, v in by_cap.items()},
            "bytes_per_launch": read_b, "writeback_bytes_per_launch": write_b, "launches": launches}


# the other workloads, timed over their whole horizon beside the headline
DETAIL_WORKLOADS = ("cfg1", "cfg2", "cfg3", "cfg4", "cfg5")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed steps (default: the workload's T)")
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="cfg4")
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds for the oracle baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the runs of the other workloads reported under detail.workloads")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the stream-ceiling measurement reported under roofline.ceiling")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="time the plain 1 GiB copy 3 times instead of 5 (for counter calibration runs)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the tuner instances are independent, so a "
              f"multi-GPU run is the same kernel on B/N instances per GPU (got --gpus {args.gpus})",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from agft_workloads import get_workload

    wl = get_workload(args.workload)
    K = wl.T if args.steps is None else args.steps
    W = args.warmup
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    # the headline's draws serve its own run over the whole horizon too
    from agft_workloads import exogenous
    draws = exogenous(wl, T=max(K, W, wl.T if wl.name in DETAIL_WORKLOADS else 1, 1))
    head = measure(wl, K, W, dev, draws=draws)
    copy_gbs = copy_rate(dev, 3 if args.calibrate_copy else 5)
    torch.cuda.synchronize()
    # the stream ceiling right after the headline's run and again with a
    # second of idle before each cap: a busy device settles a few percent
    # below the rate it starts at and recovers within half a second, so the
    # step kernel is compared with the faster of the two (run before the
    # headline, the ceiling's own load would slow the headline down)
    ceil_busy = ceil_idle = None
    ceil_error = None
    if not args.no_ceiling:
        # a side measurement: if it cannot run, the line says why and stands
        try:
            ceil_busy = stream_ceiling(wl)
            ceil_idle = stream_ceiling(wl, rest_s=1.0)
        except (OSError, RuntimeError) as exc:
            ceil_busy = ceil_idle = None
            ceil_error = str(exc)
            log(f"[bench] stream ceiling not measured: {exc}")
    traffic = counter_traffic(wl.name, steps=K, warmup=W)

    res = {
        "metric": "bandit decision-steps/sec (instances x steps) + achieved HBM GB/s vs peak",
        "value": head["value"],
        "unit": "decision-steps/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded load traces, closed-form energy-delay reward)",
        "config": {"workload": f"{wl.name}: {wl.description}", "instances": wl.B, "arms": wl.K,
                   "context_dim": wl.d, "steps_per_run": wl.T, "parallelism": "none (1 GPU)"},
        "roofline": {"bound": "hbm", "achieved": head["achieved_gbs"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": head["frac"], "traffic": traffic,
                     "traffic_window": (f"HBM bytes per step-kernel launch averaged over the {K} timed steps "
                                        f"of {wl.name} (the first {K} from a fresh state), from per-step "
                                        f"rocprofv3 counters on this kernel source"
                                        if traffic is not None else None),
                     "byte_model": byte_model(wl)},
        "detail": {k: head[k] for k in ("step_kernel_avg_ms", "step_kernel_median_ms", "step_kernel_share",
                                        "ms_per_step_fused",
                                        "algorithmic_bytes_per_launch", "mean_scored_arms",
                                        "mean_active_arms_after_step", "exploiting_fraction", "wall_s")},
    }
    res["detail"]["device_copy_gbs"] = copy_gbs
    # how agft_step launches the headline's step kernel (the first rounds of a
    # workload with the switch take the exploring width)
    from paper_2508_01744_amd import launch_shape, workload_config
    res["detail"]["launch_shape"] = launch_shape(workload_config(wl))
    if ceil_error is not None:
        res["roofline"]["ceiling"] = {"error": ceil_error}
    if ceil_busy is not None:
        c0, c1 = ceil_busy, ceil_idle
        rw = max(c0["read_writeback_gbs"], c1["read_writeback_gbs"])
        res["roofline"]["ceiling"] = {
            "read_gbs": max(c0["read_gbs"], c1["read_gbs"]), "read_writeback_gbs": rw,
            "achieved_over_read_writeback": head["achieved_gbs"] / rw,
            "after_headline": {k: c0[k] for k in ("read_gbs", "read_writeback_gbs", "read_cap",
                                                   "read_writeback_cap", "by_cap")},
            "after_idle": {k: c1[k] for k in ("read_gbs", "read_writeback_gbs", "read_cap",
                                              "read_writeback_cap", "by_cap")},
            "what": (f"the step's traffic without its arithmetic on {wl.name}'s record layout "
                     f"({c0['bytes_per_launch'] / wl.B:.0f} B read per instance, one "
                     f"{c0['writeback_bytes_per_launch'] / wl.B:.0f} B record written back), one workgroup "
                     f"per instance, non-temporal loads and stores; average of {c0['launches']} launches "
                     f"at each cap on workgroups per compute unit in {list(CEILING_CAPS)} (0: none; "
                     f"durations in us by cap), the fastest kept; measured right after the headline run "
                     f"and again with 1 s of idle before each cap, the faster of the two reported")}
    if not args.no_workloads:
        runs, ceilings = {}, {}
        if "ceiling" in res["roofline"] and "read_writeback_gbs" in res["roofline"]["ceiling"]:
            ceilings[wl.name] = res["roofline"]["ceiling"]["read_writeback_gbs"]
        for name in DETAIL_WORKLOADS:
            w2 = get_workload(name)
            if name == wl.name and args.steps is None:
                runs[name] = head
            else:
                runs[name] = measure(w2, w2.T, W, dev, log_prefix="[bench detail]",
                                     draws=draws if name == wl.name else None)
            # the stream ceiling on this workload's layout, as for the headline
            # (the faster of right after its run and rested); not for a single
            # instance, whose launch is all latency
            if not args.no_ceiling and name not in ceilings and w2.B > 1:
                try:
                    c0 = stream_ceiling(w2)
                    c1 = stream_ceiling(w2, rest_s=0.5)
                    ceilings[name] = max(c0["read_writeback_gbs"], c1["read_writeback_gbs"])
                except (OSError, RuntimeError) as exc:
                    log(f"[bench detail] {name}: stream ceiling not measured: {exc}")
        res["detail"]["workloads"] = {
            name: {"steps": r["steps"], "decision_steps_per_s": r["value"], "ms_per_step": r["ms_per_step"],
                   "decision_steps_per_s_fused": r["value_fused"], "ms_per_step_fused": r["ms_per_step_fused"],
                   "step_kernel_avg_ms": r["step_kernel_avg_ms"], "achieved_gbs": r["achieved_gbs"],
                   "frac": r["frac"], "mean_scored_arms": r["mean_scored_arms"],
                   "ceiling_read_writeback_gbs": ceilings.get(name),
                   "of_ceiling": r["achieved_gbs"] / ceilings[name] if name in ceilings else None}
            for name, r in runs.items()}
        res["detail"]["workloads_note"] = ("each workload timed over its whole horizon from a fresh state, "
                                           "step and environment kernels, inputs resident; *_fused: the same "
                                           "steps through agft_sim_step (the environment in the step kernel's "
                                           "epilogue, one launch per step, up to 8,192 instances; the step "
                                           "and environment kernels above); frac = algorithmic bytes per "
                                           "step-kernel launch over its average duration, of 8 TB/s; "
                                           "of_ceiling = the same rate over the stream ceiling's "
                                           "read-plus-write-back rate on the workload's record layout "
                                           "(measured as for the headline; the headline's own for its "
                                           "workload; none for a single instance)")
    if not args.no_cpu_baseline:
        log("[bench] timing the fp64 oracle on the host")
        base = cpu_baseline(wl, args.cpu_budget)
        # one thread over the same steps (the step mix changes as arms are
        # pruned) on a third of one thread's share of the instances
        one = cpu_baseline(wl, args.cpu_budget, threads=1, max_steps=base["steps"],
                           n_max=max(1, base["n"] // (3 * base["cores"])))
        res["cpu_baseline"] = {k: base[k] for k in ("value", "unit", "cores", "kind", "sample")}
        res["detail"]["cpu_oracle_1thread"] = {k: one[k] for k in ("value", "unit", "cores", "sample")}
        res["detail"]["host_cpu"] = host_cpu()
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
