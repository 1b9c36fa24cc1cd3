"""Seeded synthetic inputs for the batched AGFT tuner simulator.

This package holds the five workload configurations and the seeded
generators of exogenous load traces.  It contains none of the method's
arithmetic (no LinUCB scoring or update, no energy-delay model): it only
defines sizes, constants and random draws that both the GPU path and the
CPU oracle consume as inputs.
"""
from .configs import (WORKLOADS, ENV, Workload, get_workload, arm_values, with_paper_pruning,
                      with_exploitation, with_refinement, with_rule_one_reevaluated, PAPER_PRUNING)
from .traces import exogenous, probe_instances

__all__ = ["WORKLOADS", "ENV", "Workload", "get_workload", "arm_values", "with_paper_pruning",
           "with_exploitation", "with_refinement", "with_rule_one_reevaluated",
           "PAPER_PRUNING",
           "exogenous", "probe_instances"]
