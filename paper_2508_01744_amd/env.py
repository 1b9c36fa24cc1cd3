"""Python front end of the GPU serving-environment simulator (agft_sim.h)."""
import ctypes

import torch

from . import _lib as L


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def env_config(wl, env_constants, T=None, B=None):
    """agft_env_config from a workload and the environment constants."""
    c = env_constants
    cfg = L.agft_env_config()
    cfg.B = int(wl.B if B is None else B)
    cfg.K, cfg.d = int(wl.K), int(wl.d)
    cfg.T = int(wl.T if T is None else T)
    for name in ("P0", "c", "l0", "a", "b", "lat_min", "f_lo", "f_hi", "f_init", "tpot_div"):
        setattr(cfg, name, float(c[name]))
    cfg.drift = float(wl.drift)
    for name in ("svc_lo", "svc_hi", "svc_init", "q_cap", "run_cap"):
        setattr(cfg, name, int(c[name]))
    for j in range(7):
        cfg.mu[j] = float(c["mu"][j])
        cfg.sd[j] = float(c["sd"][j])
    return cfg


class GpuEnv:
    """B simulated serving nodes; arrivals/noise are [T+1][B] device tensors."""

    def __init__(self, cfg, arrivals, noise, stream=None):
        self.cfg = cfg
        self.B, self.d, self.T = cfg.B, cfg.d, cfg.T
        dev = arrivals.device
        if arrivals.dtype != torch.int32 or noise.dtype != torch.float32:
            raise ValueError("arrivals must be int32 and noise float32")
        if tuple(arrivals.shape) != (self.T + 1, self.B) or tuple(noise.shape) != (self.T + 1, self.B):
            raise ValueError("arrivals and noise must be [T+1][B]")
        self.arrivals = arrivals.contiguous()
        self.noise = noise.contiguous()
        self.nbytes = L.agft_env_state_bytes(cfg)
        if self.nbytes == 0:
            raise ValueError("invalid environment configuration")
        # zeroed so that the alignment gaps between regions are deterministic
        self.state = torch.zeros(self.nbytes, dtype=torch.uint8, device=dev)
        self.ctx = torch.empty(self.B, self.d, dtype=torch.float32, device=dev)
        self.reward = torch.empty(self.B, dtype=torch.float32, device=dev)
        self.stream = stream if stream is not None else torch.cuda.current_stream(dev)

    def _s(self):
        return ctypes.c_void_p(self.stream.cuda_stream)

    def reset(self):
        L.check("agft_env_reset", L.agft_env_reset(self.cfg, _ptr(self.state), self.nbytes,
                                                   _ptr(self.arrivals), _ptr(self.noise),
                                                   _ptr(self.ctx), self._s()))
        return self.ctx

    def step(self, t, action):
        L.check("agft_env_step", L.agft_env_step(self.cfg, _ptr(self.state), self.nbytes, int(t),
                                                 _ptr(action), _ptr(self.arrivals),
                                                 _ptr(self.noise), _ptr(self.reward),
                                                 _ptr(self.ctx), self._s()))
        return self.reward, self.ctx

    def fused_step(self, tuner, action, scores=None):
        """One decision of tuner (agft_step) and this environment's response
        to it (agft_sim_step: one launch up to 8,192 instances, the step and
        environment kernels above): self.ctx and self.reward hold x_t and
        r_{t-1} on entry and x_{t+1} and r_t on return."""
        tuner._check(action, (self.B,), torch.int32)
        tuner._check(scores, (self.B, 2, tuner.K), torch.float32)
        L.check("agft_sim_step", L.agft_sim_step(tuner.h, self.cfg, _ptr(self.state), self.nbytes,
                                                 _ptr(self.arrivals), _ptr(self.noise), _ptr(self.ctx),
                                                 _ptr(self.reward), _ptr(action), _ptr(scores)))
        return self.reward, self.ctx
