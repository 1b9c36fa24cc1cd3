"""CPU fp64 oracle of the AGFT bandit step and of the synthetic serving
environment.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.  It shares no code
with the GPU path; both read their inputs from agft_workloads.
"""
from .oracle import Oracle, load_library, build_library
from .env import Env
from .run import run_closed_loop

__all__ = ["Oracle", "Env", "run_closed_loop", "load_library", "build_library"]
