"""Seeded synthetic workloads for the SFS TTFT estimator and router.

This package only draws inputs: instance snapshots (remaining prefill, predicted
remaining decode, context), query traces (arrival time, prompt length, predicted
decode length), accuracy and cost predictions, and routing weights.  It holds none
of the estimator's or router's arithmetic, so both the CPU oracle and the HIP path
can consume the same arrays without sharing any code that computes results.
"""

from .configs import CONFIGS, config_names, get_config
from .gen import Workload, make_workload, make_tiny_workload

__all__ = ["CONFIGS", "config_names", "get_config", "Workload", "make_workload",
           "make_tiny_workload"]
