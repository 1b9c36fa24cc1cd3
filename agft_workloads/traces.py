"""Seeded exogenous load traces for the tuner simulator.

Every instance i of workload c draws from its own generator,
numpy.random.default_rng([2508, 1744, c, i]), so any subset of instances (the
probe instances of a full-size run) can be regenerated alone and matches the
full batch exactly.  Draw order per instance:

1. trace parameters (family dependent, below);
2. the family's per-window innovations;
3. Poisson arrival counts n_w ~ Poisson(rate_w), w = 0..T;
4. latency noise eta_w ~ N(0, noise_sd^2), rounded to float32.

Families (window w = 0..T, one window per decision, window 0 is the warm-up
window run before the first decision):

* "sinusoid_ar1": rate_w = max(0.5, 10 + 6 sin(2 pi w / 600) + y_w),
  y_w = 0.9 y_{w-1} + 1.5 e_w, e_w ~ N(0, 1);
* "ar1_uniform_mean": m ~ U(0.5, 20); rate_w = max(0.1, m + y_w),
  y_w = 0.9 y_{w-1} + 0.2 m e_w;
* "onoff": on-rate ~ U(10, 20), off-rate ~ U(0.5, 3), initial state on with
  probability 1/2, and the state flips in window w when u_w < 0.02,
  u_w ~ U(0, 1).

These stand in for the production LLM inference traces the paper drives its
tuner with (hour-scale volatility with large dispersion and bursts, Sec. 2.4),
which are not available here.
"""
import numpy as np
from scipy.signal import lfilter

from .configs import ENV, Workload

SEED = (2508, 1744)


def _rates(wl: Workload, rng, W: int) -> np.ndarray:
    w = np.arange(W, dtype=np.float64)
    if wl.trace == "sinusoid_ar1":
        e = rng.standard_normal(W)
        y = lfilter([1.5], [1.0, -0.9], e)
        return np.maximum(0.5, 10.0 + 6.0 * np.sin(2.0 * np.pi * w / 600.0) + y)
    if wl.trace == "ar1_uniform_mean":
        m = rng.uniform(0.5, 20.0)
        e = rng.standard_normal(W)
        y = lfilter([0.2 * m], [1.0, -0.9], e)
        return np.maximum(0.1, m + y)
    if wl.trace == "onoff":
        on_rate = rng.uniform(10.0, 20.0)
        off_rate = rng.uniform(0.5, 3.0)
        s0 = rng.random() < 0.5
        flips = rng.random(W) < 0.02
        state = np.logical_xor(s0, np.cumsum(flips) % 2 == 1)
        return np.where(state, on_rate, off_rate)
    raise ValueError(f"unknown trace family {wl.trace!r}")


def exogenous(wl: Workload, instances=None, T: int = None):
    """Arrival counts and latency noise for windows 0..T of the given instances.

    Returns (arrivals int32 [T+1][n], noise float32 [T+1][n]), time-major, where
    n = len(instances) (default: all B instances).
    """
    if instances is None:
        instances = range(wl.B)
    instances = [int(i) for i in instances]
    T = wl.T if T is None else int(T)
    W = T + 1
    arrivals = np.empty((W, len(instances)), dtype=np.int32)
    noise = np.empty((W, len(instances)), dtype=np.float32)
    sd = ENV["noise_sd"]
    for col, i in enumerate(instances):
        if not 0 <= i < wl.B:
            raise ValueError(f"instance {i} outside [0, {wl.B})")
        rng = np.random.default_rng([SEED[0], SEED[1], wl.cfg_id, i])
        rate = _rates(wl, rng, W)
        arrivals[:, col] = rng.poisson(rate)
        noise[:, col] = (rng.standard_normal(W) * sd).astype(np.float32)
    return arrivals, noise


def probe_instances(B: int, n: int = 64):
    """Instances recorded in full-size runs: evenly strided, first and last included."""
    if B <= n:
        return list(range(B))
    return sorted(set(int(round(v)) for v in np.linspace(0, B - 1, n)))
