"""The five tuner-simulator workloads and the constants of the synthetic
serving environment.

Each workload is B independent tuner instances, K frequency arms, a context of
d features and a horizon of T decisions.  The paper's own controller sees one
7-feature context per sub-second window (Sec. 4.1) and picks among
fine-grained frequency steps (Sec. 3.2, Sec. 4.4); the batched instances stand
in for many such controllers at once.

Environment constants (power/latency closed form, feature normalisation) are
data: both the GPU simulator and the CPU oracle read them from here and each
implements the closed form on its own.
"""
from dataclasses import dataclass
import math


@dataclass(frozen=True)
class Workload:
    name: str
    cfg_id: int          # seed component and stable identifier (1..5)
    B: int               # independent tuner instances
    K: int               # frequency arms, uniform on [f_lo, f_hi]
    d: int               # context dimension (8, 16 or 32)
    T: int               # decisions per run
    lam: float           # ridge prior: A_k(0) = lam * I
    alpha0: float        # exploration weight
    alpha_sched: int     # 0: alpha_t = alpha0; 1: alpha_t = alpha0 / sqrt(t + 1)
    prune: int           # rule mask: 1 drop arm k when UCB_k < max_j LCB_j (every
                         # `period` steps); 2 extreme-frequency, 4 historical-
                         # performance, 8 cascade pruning (Sec. 4.3)
    period: int          # prune evaluated at t > 0 with t % period == 0
    trace: str           # load-trace family, see traces.py
    drift: float = 0.0   # power/latency coefficients b, c scale to (1 + drift) at t = T - 1
    description: str = ""
    # rule 1 removes arms for good (1), or is re-evaluated over the whole
    # action space at each of its steps (0: the non-sticky reading)
    prune_sticky: int = 1
    # the paper's pruning heuristics (rule bits 2, 4, 8; Sec. 4.3): the example
    # values the paper gives, plus a reading of the unstated ones
    # (tolerance multiplier and the minimum number of compared arms)
    ext_rounds: int = 60
    ext_min_n: int = 3
    ext_thr: float = -1.2
    hist_after: int = 30
    hist_min_n: int = 6
    hist_kappa: float = 1.0
    hist_min_arms: int = 3
    # switch to greedy exploitation once a Page-Hinkley test finds the reward
    # sequence stable (Sec. 4.2, Eq. 2); the paper names the test but none of
    # its constants, except a maturity threshold of 100 rounds (Sec. 4.4)
    exploit: int = 0
    ph_delta: float = 0.05
    ph_lambda: float = 5.0
    ph_window: int = 100
    ph_min_rounds: int = 100
    # mixed-maturity refinement of the action space (Sec. 4.4): one arm step
    # of the K-arm grid plays the paper's 15 MHz step, so its +-150 MHz window
    # is +-10 arms (21 arms) and the coarse starting grid takes every 10th arm;
    # maturity after 100 rounds and 4 samples for the statistical anchor are
    # the paper's example values; the refinement period is unstated
    refine: int = 0
    refine_period: int = 50
    refine_stride: int = 10
    refine_half: int = 10
    refine_mature: int = 100
    refine_min_n: int = 4

    @property
    def arm_record_floats(self) -> int:
        """Floats of per-arm bandit state the GPU path keeps (theta + packed factor)."""
        return self.d + self.d * (self.d + 1) // 2

    @property
    def cascade_k(self) -> int:
        """Arms whose clock is below half of the top clock (cascade rule)."""
        return sum(1 for f in arm_values(self.K) if f < 0.5 * ENV["f_hi"])

    def heuristics(self) -> dict:
        return dict(ext_rounds=self.ext_rounds, ext_min_n=self.ext_min_n, ext_thr=self.ext_thr,
                    hist_after=self.hist_after, hist_min_n=self.hist_min_n,
                    hist_kappa=self.hist_kappa, hist_min_arms=self.hist_min_arms,
                    cascade_k=self.cascade_k)

    def page_hinkley(self) -> dict:
        return dict(ph_delta=self.ph_delta, ph_lambda=self.ph_lambda, ph_window=self.ph_window,
                    ph_min_rounds=self.ph_min_rounds)

    def refinement(self) -> dict:
        return dict(refine_period=self.refine_period, refine_stride=self.refine_stride,
                    refine_half=self.refine_half, refine_mature=self.refine_mature,
                    refine_min_n=self.refine_min_n)

    def alpha_at(self, t: int) -> float:
        if self.alpha_sched == 0:
            return self.alpha0
        return self.alpha0 / math.sqrt(t + 1.0)


WORKLOADS = {
    1: Workload("cfg1", 1, B=1, K=16, d=8, T=10_000, lam=1.0, alpha0=1.0,
                alpha_sched=0, prune=0, period=50, trace="sinusoid_ar1",
                description="1 instance, 16 arms, d=8, 10,000 steps, alpha=1, no pruning"),
    2: Workload("cfg2", 2, B=4096, K=64, d=8, T=2000, lam=1.0, alpha0=0.5,
                alpha_sched=0, prune=0, period=50, trace="ar1_uniform_mean",
                description="4,096 instances, 64 arms, d=8, 2,000 steps, alpha=0.5, no pruning"),
    3: Workload("cfg3", 3, B=16_384, K=128, d=16, T=1000, lam=1.0, alpha0=0.5,
                alpha_sched=0, prune=1, period=50, trace="ar1_uniform_mean",
                description="16,384 instances, 128 arms, d=16, 1,000 steps, pruning every 50"),
    4: Workload("cfg4", 4, B=65_536, K=128, d=16, T=500, lam=1.0, alpha0=0.5,
                alpha_sched=0, prune=1, period=50, trace="onoff",
                description="65,536 instances, 128 arms, d=16, 500 steps, bursty on/off "
                            "traces, pruning every 50, alpha=0.5"),
    5: Workload("cfg5", 5, B=1024, K=256, d=32, T=2000, lam=1.0, alpha0=1.0,
                alpha_sched=1, prune=1, period=50, trace="ar1_uniform_mean", drift=0.3,
                description="1,024 instances, 256 arms, d=32, 2,000 steps, drifting "
                            "reward model, alpha_t = 1/sqrt(t+1), pruning every 50"),
}


PAPER_PRUNING = 2 | 4 | 8


def with_paper_pruning(wl: Workload) -> Workload:
    """The same workload with the paper's pruning heuristics added to its rules."""
    d = dict(wl.__dict__)
    d["prune"] = wl.prune | PAPER_PRUNING
    d["name"] = wl.name + "p"
    d["description"] = wl.description + ", plus the paper's extreme/historical/cascade pruning"
    return Workload(**d)


def with_exploitation(wl: Workload) -> Workload:
    """The same workload with the Page-Hinkley switch to greedy exploitation."""
    d = dict(wl.__dict__)
    d["exploit"] = 1
    d["name"] = wl.name + "e"
    d["description"] = wl.description + ", plus the switch to greedy exploitation"
    return Workload(**d)


def with_rule_one_reevaluated(wl: Workload) -> Workload:
    """The same workload with rule 1 re-evaluated over every arm at each of
    its steps instead of removing arms for good."""
    d = dict(wl.__dict__)
    d["prune_sticky"] = 0
    d["name"] = wl.name + "n"
    d["description"] = wl.description + ", rule 1 re-evaluated over every arm at each of its steps"
    return Workload(**d)


def with_refinement(wl: Workload) -> Workload:
    """The same workload with the mixed-maturity refinement of the action space."""
    d = dict(wl.__dict__)
    d["refine"] = 1
    d["name"] = wl.name + "r"
    d["description"] = wl.description + ", plus the mixed-maturity refinement"
    return Workload(**d)


def get_workload(cfg, **overrides) -> Workload:
    """Workload by id (1..5) or name ("cfg4"), optionally with fields replaced
    (smaller B or T for quick parity cases)."""
    suffix = ""
    if isinstance(cfg, str):
        body = cfg.replace("cfg", "")
        suffix = body.lstrip("0123456789")
        cfg = int(body[:len(body) - len(suffix)])
        if set(suffix) - set("pern"):
            raise ValueError(f"unknown workload suffix {suffix!r} (p: paper pruning, "
                             f"e: exploitation, r: refinement, n: rule 1 re-evaluated)")
        if "n" in suffix and "p" in suffix:
            raise ValueError("the paper's rules remove arms for good: no re-evaluated rule 1 beside them")
    wl = WORKLOADS[cfg]
    if "p" in suffix:
        wl = with_paper_pruning(wl)
    if "e" in suffix:
        wl = with_exploitation(wl)
    if "r" in suffix:
        wl = with_refinement(wl)
    if "n" in suffix:
        wl = with_rule_one_reevaluated(wl)
    if overrides:
        d = dict(wl.__dict__)
        d.update(overrides)
        wl = Workload(**d)
    return wl


# Constants of the synthetic serving environment.  Energy-delay product is
# energy x delay (Sec. 2.3); per window, energy = power x latency and delay =
# latency, so EDP = power * latency^2.  Power rises with the cube of the
# normalised clock, latency falls with it in proportion to load; the product
# has an interior minimum that moves up with load, the U-shape of Fig. 6.
ENV = dict(
    P0=0.3, c=0.7,          # power(f) = P0 + c f^3  (power(1) = 1)
    l0=1.0, a=0.5, b=0.05,  # latency(f) = l0 (a + b n / f) + noise
    lat_min=0.05,           # latency floor
    noise_sd=0.02,          # latency noise standard deviation
    f_lo=0.2, f_hi=1.0,     # normalised arm grid
    f_init=0.6,             # clock of the warm-up window before the first decision
    svc_lo=5, svc_hi=25,    # integer service capacity (requests/window) at f_lo, f_hi
    svc_init=15,            # service capacity at f_init
    q_cap=200,              # waiting-queue cap (requests beyond it are dropped)
    run_cap=64,             # concurrency cap
    tpot_div=8.0,           # TPOT = latency / tpot_div
    # z-score constants of the 7 raw features
    # [arrivals, log1p(queue), running, log(TTFT), TPOT, util, clock],
    # rounded from the feature means and deviations of random-arm runs of
    # the three trace families, so that features are O(1)
    mu=(9.0, 1.6, 23.0, 0.9, 0.18, 0.54, 0.6),
    sd=(8.0, 2.0, 25.0, 1.5, 0.125, 0.38, 0.23),
)


def arm_values(K: int):
    """Normalised clock of every arm: uniform steps over [f_lo, f_hi]."""
    lo, hi = ENV["f_lo"], ENV["f_hi"]
    if K == 1:
        return [hi]
    return [lo + (hi - lo) * k / (K - 1) for k in range(K)]
