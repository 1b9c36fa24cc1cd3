"""AGFT's contextual-bandit frequency tuner as a batched MI355X (gfx950) step.

The hot path lives in libagft.so (HIP kernels behind the C ABI of
include/agft.h and include/agft_sim.h); this package only binds it.
"""
from ._lib import LIB_PATH, AgftError, lib
from .tuner import Tuner, launch_shape, make_config, workload_config
from .env import GpuEnv, env_config
from .sim import run_closed_loop

__all__ = ["LIB_PATH", "AgftError", "lib", "Tuner", "launch_shape", "make_config", "workload_config",
           "GpuEnv", "env_config", "run_closed_loop"]
