"""Synthetic analogs of the paper's quality experiments (Sec. 5), run on the
batched GPU simulator.

The paper measures its controller on a real server: energy, EDP, TTFT and
TPOT against the driver's default clocks before and after convergence
(Sec. 5.3), the learned clock against an offline optimum per workload type,
two ablations (a coarser action space, no pruning; Sec. 5.4), and the rolling
mean and spread of the reward as learning proceeds.  Here the same quantities
come from the closed-form serving model that drives the tuner instances:

* per window, from the context the environment reports after decision t
  (features 3 and 4: log TTFT and TPOT, z-scored), latency = TPOT * tpot_div,
  power = P0 + c_w f^3, energy = power * latency, EDP = energy * latency;
* "default clocks" is the same environment run with every decision at the
  top arm;
* the convergence point of an instance is its switch to exploitation when
  the workload has the switch, otherwise half of the run;
* the offline optimum of an instance is the arm with the best noise-free
  reward (EDP relative to the top clock's at the same load, the quantity the
  tuner learns) summed over its post-convergence windows; the online choice is
  the arm it chose most often in those windows;
* "no-grain" keeps the coarse starting grid (every 10th arm) for the whole
  run; "no pruning" clears every pruning rule.

Every step of the method runs in the tuner's and the environment's kernels;
this module only drives them and reduces what they report with torch.

    python -m paper_2508_01744_amd.experiments --workload cfg3per [--instances 4096]
"""
import argparse
import json
import sys

import torch

from agft_workloads import ENV, exogenous, get_workload
from .env import GpuEnv, env_config
from .tuner import Tuner

METRICS = ("energy", "edp", "ttft", "tpot")


def arm_clocks(K, device):
    if K == 1:
        return torch.full((1,), ENV["f_hi"], dtype=torch.float64, device=device)
    k = torch.arange(K, dtype=torch.float64, device=device)
    return ENV["f_lo"] + (ENV["f_hi"] - ENV["f_lo"]) * k / (K - 1)


def drift_scale(wl, t):
    """Scale of b and c in the window of decision t (0-based)."""
    return 1.0 + wl.drift * (t / (wl.T - 1) if wl.T > 1 else 0.0)


def noise_free_edp(n, f, scale):
    """Noise-free EDP of windows with arrivals n [..., 1] at clocks f [K]."""
    b, c = ENV["b"] * scale, ENV["c"] * scale
    lat = torch.clamp(ENV["l0"] * (ENV["a"] + b * n / f), min=ENV["lat_min"])
    return (ENV["P0"] + c * f ** 3) * lat * lat


def window_metrics(ctx, clock, scale):
    """Energy, EDP, TTFT, TPOT of the window just run, from its context."""
    mu, sd = ENV["mu"], ENV["sd"]
    ttft = torch.exp(ctx[:, 4].double() * sd[3] + mu[3])
    tpot = ctx[:, 5].double() * sd[4] + mu[4]
    lat = tpot * ENV["tpot_div"]
    energy = (ENV["P0"] + ENV["c"] * scale * clock ** 3) * lat
    return dict(energy=energy, edp=energy * lat, ttft=ttft, tpot=tpot)


class _Acc:
    """Per-instance sums for the mean and coefficient of variation of each
    metric over a masked subset of the windows."""

    def __init__(self, B, device):
        z = lambda: torch.zeros(B, dtype=torch.float64, device=device)
        self.n = z()
        self.s = {m: z() for m in METRICS}
        self.q = {m: z() for m in METRICS}

    def add(self, vals, mask):
        w = mask.double()
        self.n += w
        for m in METRICS:
            self.s[m] += w * vals[m]
            self.q[m] += w * vals[m] * vals[m]

    def summary(self):
        ok = self.n > 1
        out = {}
        for m in METRICS:
            mean = self.s[m][ok] / self.n[ok]
            var = torch.clamp(self.q[m][ok] / self.n[ok] - mean * mean, min=0.0)
            out[m] = dict(mean=float(mean.mean()), cv=float((var.sqrt() / mean).mean()))
        out["instances"] = int(ok.sum())
        return out


def run(wl, device="cuda", baseline=False, window=50, checkpoints=10):
    """Run wl closed loop.  With baseline, a second environment on the same
    draws runs every window at the top clock, and its windows are summarised
    with the tuner run's convergence split.  Returns pre- and
    post-convergence summaries, the convergence rounds, the online and
    offline arms per instance, and rolling reward statistics."""
    dev = torch.device(device)
    B, K, T = wl.B, wl.K, wl.T
    arr, noi = exogenous(wl)
    arr_d = torch.as_tensor(arr, device=dev)
    noi_d = torch.as_tensor(noi, device=dev)
    env = GpuEnv(env_config(wl, ENV), arr_d, noi_d)
    env_b = GpuEnv(env_config(wl, ENV), arr_d, noi_d) if baseline else None
    clocks = arm_clocks(K, dev)
    tuner = Tuner.from_workload(wl, device=dev)
    view = tuner.view()
    action = torch.empty(B, dtype=torch.int32, device=dev)
    top = torch.full((B,), K - 1, dtype=torch.int32, device=dev)
    acc = {ph: _Acc(B, dev) for ph in ("pre", "post", "default_pre", "default_post")}
    counts = torch.zeros(B, K, dtype=torch.int64, device=dev)
    offline = torch.zeros(B, K, dtype=torch.float64, device=dev)
    conv = torch.full((B,), T // 2, dtype=torch.int64, device=dev)
    ring = torch.zeros(window, B, dtype=torch.float64, device=dev)
    rolling = []
    x = env.reset()
    if env_b is not None:
        env_b.reset()
    r = None
    for t in range(T):
        tuner.step(x, r, action)
        if wl.exploit:
            mode = view["mode"].long()
            converged = mode >= 0
            conv = torch.where(converged, mode, torch.full_like(mode, T))
        else:
            converged = torch.full((B,), t >= T // 2, dtype=torch.bool, device=dev)
        a = action.long().clamp(min=0)
        scale = drift_scale(wl, t)
        r, x = env.step(t, action)
        vals = window_metrics(x, clocks[a], scale)
        acc["pre"].add(vals, ~converged)
        acc["post"].add(vals, converged)
        if env_b is not None:
            _, xb = env_b.step(t, top)
            vb = window_metrics(xb, clocks[top.long()], scale)
            acc["default_pre"].add(vb, ~converged)
            acc["default_post"].add(vb, converged)
        counts += torch.nn.functional.one_hot(a, K) * converged.long()[:, None]
        n = arr_d[t + 1].double()[:, None]
        rel = noise_free_edp(n, clocks[None, :], scale) / noise_free_edp(n, clocks[-1:], scale)
        offline += rel * converged.double()[:, None]
        ring[t % window] = r.double()
        if (t + 1) % max(1, T // checkpoints) == 0 and t + 1 >= window:
            rolling.append(dict(round=t + 1, mean=float(ring.mean(dim=0).mean()),
                                std=float(ring.std(dim=0).mean())))
    torch.cuda.synchronize(dev)
    out = dict(convergence=conv, has_post=counts.sum(dim=1) > 0, online=counts.argmax(dim=1),
               offline=offline.argmin(dim=1), rolling=rolling, mean_load=arr_d[1:].double().mean(dim=0))
    for ph, a_ in acc.items():
        if baseline or not ph.startswith("default"):
            out[ph] = a_.summary()
    return out


def _diff(a, b):
    return 100.0 * (a - b) / b


def frequency_table(res, wl, quantiles=5):
    """Offline versus online clock per quintile of mean load (the analog of
    the paper's per-workload comparison)."""
    dev = res["online"].device
    clocks = arm_clocks(wl.K, dev)
    sel = res["has_post"]
    load = res["mean_load"][sel]
    f_on, f_off = clocks[res["online"][sel]], clocks[res["offline"][sel]]
    order = torch.argsort(load)
    rows = []
    for q in range(quantiles):
        idx = order[q * len(order) // quantiles:(q + 1) * len(order) // quantiles]
        if len(idx) == 0:
            continue
        on, off = float(f_on[idx].mean()), float(f_off[idx].mean())
        rows.append(dict(load=float(load[idx].mean()), offline=off, online=on, deviation=_diff(on, off),
                         abs_deviation=float((100.0 * (f_on[idx] - f_off[idx]).abs() / f_off[idx]).mean())))
    return rows


def ablation_variants(wl):
    """The coarse grid only ("no-grain") and no pruning rule ("no pruning")."""
    d = dict(wl.__dict__)
    return {"no-grain": type(wl)(**dict(d, refine=1, refine_stride=10, refine_period=wl.T + 1)),
            "no pruning": type(wl)(**dict(d, prune=0))}


def report(name, B=None, T=None, device="cuda"):
    over = {k: v for k, v in (("B", B), ("T", T)) if v is not None}
    wl = get_workload(name, **over)
    full = run(wl, device=device, baseline=True)
    out = dict(workload=wl.name, description=wl.description, instances=wl.B, steps=wl.T, arms=wl.K)
    out["vs_default"] = {ph: {m: dict(agft=full[ph][m]["mean"], default=full["default_" + ph][m]["mean"],
                                      diff=_diff(full[ph][m]["mean"], full["default_" + ph][m]["mean"]))
                              for m in METRICS} for ph in ("pre", "post")}
    out["frequency"] = frequency_table(full, wl)
    out["ablation"] = {"full": {m: full["post"][m] for m in METRICS}}
    for label, v in ablation_variants(wl).items():
        res = run(v, device=device)
        out["ablation"][label] = {m: res["post"][m] for m in METRICS}
    out["rolling_reward"] = full["rolling"]
    conv = full["convergence"]
    switched = conv < wl.T
    out["convergence_round"] = float(conv[switched].double().mean()) if bool(switched.any()) else None
    out["switched_fraction"] = float(switched.double().mean()) if wl.exploit else None
    return out


def markdown(rep):
    L = [f"### {rep['workload']}: {rep['description']}", ""]
    if rep.get("convergence_round") is not None:
        L.append(f"Mean convergence (switch) round {rep['convergence_round']:.0f}; "
                 f"{100 * rep['switched_fraction']:.0f}% of instances switched.")
        L.append("")
    for ph, title in (("pre", "before convergence"), ("post", "after convergence")):
        L += [f"Against the top clock, {title}:", "", "| metric | AGFT | top clock | diff |", "|---|---|---|---|"]
        for m in METRICS:
            v = rep["vs_default"][ph][m]
            L.append(f"| {m} | {v['agft']:.4g} | {v['default']:.4g} | {v['diff']:+.1f}% |")
        L.append("")
    L += ["Learned versus offline-optimal clock by load quintile:", "",
          "| mean arrivals | offline f | online f | deviation | mean abs deviation |", "|---|---|---|---|---|"]
    for row in rep["frequency"]:
        L.append(f"| {row['load']:.2f} | {row['offline']:.3f} | {row['online']:.3f} | {row['deviation']:+.1f}% "
                 f"| {row['abs_deviation']:.1f}% |")
    L += ["", "Ablations, after convergence (mean, coefficient of variation):", "",
          "| variant | " + " | ".join(METRICS) + " |", "|---|" + "---|" * len(METRICS)]
    for label, row in rep["ablation"].items():
        L.append(f"| {label} | " + " | ".join(f"{row[m]['mean']:.4g} ({row[m]['cv']:.3f})" for m in METRICS)
                 + " |")
    L += ["", "Rolling reward (window 50, averaged over instances):", "", "| round | mean | std |",
          "|---|---|---|"]
    for row in rep["rolling_reward"]:
        L.append(f"| {row['round']} | {row['mean']:.4f} | {row['std']:.4f} |")
    return "\n".join(L)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--workload", default="cfg3per")
    ap.add_argument("--instances", type=int, default=None)
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--json", default=None, help="also write the report as JSON here")
    args = ap.parse_args(argv)
    rep = report(args.workload, B=args.instances, T=args.steps)
    print(markdown(rep), flush=True)
    if args.json:
        with open(args.json, "w") as fh:
            json.dump(rep, fh, indent=1)


if __name__ == "__main__":
    sys.exit(main())
