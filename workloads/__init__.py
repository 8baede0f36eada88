"""Seeded synthetic inputs for group decode attention.

This package only draws random inputs and lays them out in the paged-KV form
that both the CPU oracle and the HIP library consume. It performs none of the
attention arithmetic, so it can be shared by both sides without coupling them.
"""
from .configs import CONFIGS, config_by_id
from .gen import Workload, make_config_workload, make_workload
from .prefill import PrefillWorkload, make_prefill_workload
from .qkprep import QkPrepInputs, make_qkprep_inputs
from .rollout import make_rollout_workload

__all__ = ["CONFIGS", "config_by_id", "Workload", "make_config_workload", "make_workload",
           "PrefillWorkload", "make_prefill_workload",
           "QkPrepInputs", "make_qkprep_inputs", "make_rollout_workload"]
