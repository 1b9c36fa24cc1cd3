"""fp64 numpy model of the synthetic serving environment that feeds the tuner.

Test infrastructure only.  Written independently of the GPU simulator; both
read their constants and exogenous draws from agft_workloads.

Window w = 0..T runs at normalised clock f_w: window 0 at f_init (warm-up,
before the first decision), window t+1 at the arm chosen at decision t.  With
n = arrivals[w], eta = noise[w] and drift fraction tau_w = t / (T - 1) for the
window of decision t (0 for the warm-up window):

  b_w, c_w   = b (1 + drift tau_w), c (1 + drift tau_w)
  latency    = max(lat_min, l0 (a + b_w n / f) + eta)
  power      = P0 + c_w f^3
  EDP        = power * latency^2              (energy x delay, Sec. 2.3)
  EDP_ref    = (P0 + c_w) (l0 (a + b_w n))^2  (noise-free EDP at full clock)
  reward     = -EDP / EDP_ref                 (higher is better; -1 at full clock)
  queue      = min(q_cap, max(0, queue + n - cap))    (integers)
  running    = min(run_cap, queue + n)
  TTFT       = latency (1 + queue / cap),  TPOT = latency / tpot_div
  util       = min(1, n / cap)
  features z = ([n, log1p(queue), running, log(TTFT), TPOT, util, f] - mu) / sd

cap is the integer service capacity round(svc_lo + (svc_hi - svc_lo) k/(K-1))
of arm k (svc_init for the warm-up window).  The context of decision t is

  d = 8:  [1, z_t]
  d = 16: [1, z_t, z_{t-1}, rho_t]
  d = 32: [1, z_t, z_{t-1}, z_{t-2}, z_{t-3}, rho_t, rho_{t-1}, rho_{t-2}]

with z_w, rho_w the features and reward of window w, and windows before 0
repeating window 0.  The reward of decision t is rho_{t+1}.  An action of -1
(no decision) keeps the previous clock.

The paper prints no worked example of its reward or features, so the
constants (agft_workloads.ENV) are parity unpinned with respect to it; the
tests pin this model's structure instead (the EDP identities, the position of
its optimum, the integer capacities, the context layout).
"""
import numpy as np

from agft_workloads import ENV


class Env:
    def __init__(self, wl, arrivals, noise, T=None):
        self.wl = wl
        self.T = wl.T if T is None else int(T)
        self.arrivals = np.asarray(arrivals, dtype=np.float64)
        self.noise = np.asarray(noise, dtype=np.float64)
        if self.arrivals.shape[0] < self.T + 1:
            raise ValueError("need T+1 windows of exogenous draws")
        self.n = self.arrivals.shape[1]
        self.d = wl.d
        self.K = wl.K
        self.mu = np.array(ENV["mu"], dtype=np.float64)
        self.sd = np.array(ENV["sd"], dtype=np.float64)

    def arm_clock(self, k):
        k = np.asarray(k, dtype=np.float64)
        if self.K == 1:
            return np.full(k.shape, ENV["f_hi"])
        return ENV["f_lo"] + (ENV["f_hi"] - ENV["f_lo"]) * k / (self.K - 1)

    def arm_capacity(self, k):
        k = np.asarray(k, dtype=np.int64)
        if self.K == 1:
            return np.full(k.shape, ENV["svc_hi"], dtype=np.int64)
        p = ENV["svc_lo"] * (self.K - 1) + (ENV["svc_hi"] - ENV["svc_lo"]) * k
        q = self.K - 1
        return (2 * p + q) // (2 * q)          # round(p / q), halves up

    def _window(self, w):
        T = self.T
        tau = 0.0 if (w == 0 or T <= 1) else (w - 1) / (T - 1)
        scale = 1.0 + self.wl.drift * tau
        bw, cw = ENV["b"] * scale, ENV["c"] * scale
        n = self.arrivals[w]
        f = self.f
        cap = self.cap.astype(np.float64)
        lat = np.maximum(ENV["lat_min"], ENV["l0"] * (ENV["a"] + bw * n / f) + self.noise[w])
        power = ENV["P0"] + cw * f ** 3
        lat_ref = ENV["l0"] * (ENV["a"] + bw * n)
        reward = -(power * lat * lat) / ((ENV["P0"] + cw) * lat_ref * lat_ref)
        self.q = np.minimum(ENV["q_cap"], np.maximum(0, self.q + self.arrivals[w].astype(np.int64)
                                                     - self.cap))
        running = np.minimum(ENV["run_cap"], self.q + self.arrivals[w].astype(np.int64))
        ttft = lat * (1.0 + self.q / cap)
        tpot = lat / ENV["tpot_div"]
        util = np.minimum(1.0, n / cap)
        raw = np.stack([n, np.log1p(self.q.astype(np.float64)), running.astype(np.float64),
                        np.log(ttft), tpot, util, f], axis=1)
        z = (raw - self.mu) / self.sd
        return reward, z

    def _context(self):
        one = np.ones((self.n, 1))
        zh, rh = self.zh, self.rh        # most recent last
        if self.d == 8:
            return np.concatenate([one, zh[-1]], axis=1)
        if self.d == 16:
            return np.concatenate([one, zh[-1], zh[-2], rh[-1][:, None]], axis=1)
        if self.d == 32:
            return np.concatenate([one, zh[-1], zh[-2], zh[-3], zh[-4],
                                   rh[-1][:, None], rh[-2][:, None], rh[-3][:, None]], axis=1)
        raise ValueError("context dimension must be 8, 16 or 32")

    def reset(self):
        """Run the warm-up window; return x_0 [n][d]."""
        self.q = np.zeros(self.n, dtype=np.int64)
        self.f = np.full(self.n, ENV["f_init"])
        self.cap = np.full(self.n, ENV["svc_init"], dtype=np.int64)
        r, z = self._window(0)
        self.zh = [z, z, z, z]
        self.rh = [r, r, r]
        return self._context()

    def step(self, t, action):
        """Run window t+1 at the clock of a_t; return (r_t [n], x_{t+1} [n][d])."""
        action = np.asarray(action)
        ok = action >= 0
        safe = np.where(ok, action, 0)
        self.f = np.where(ok, self.arm_clock(safe), self.f)
        self.cap = np.where(ok, self.arm_capacity(safe), self.cap)
        r, z = self._window(t + 1)
        self.zh = self.zh[1:] + [z]
        self.rh = self.rh[1:] + [r]
        return r, self._context()
