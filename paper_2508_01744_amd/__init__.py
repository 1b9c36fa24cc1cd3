"""AGFT's contextual-bandit frequency tuner as a batched MI355X (gfx950) step.

The hot path lives in libagft.so (HIP kernels behind the C ABI of
include/agft.h and include/agft_sim.h); this package only binds it.
"""
from ._lib import LIB_PATH, AgftError, lib
from .tuner import Tuner
from .env import GpuEnv, env_config
from .sim import run_closed_loop

__all__ = ["LIB_PATH", "AgftError", "lib", "Tuner", "GpuEnv", "env_config", "run_closed_loop"]
