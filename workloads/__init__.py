"""Seeded synthetic inputs shared by the oracle side and the GPU side.

Holds the workload table, the instance builder (units, costs, CSR topology)
and the candidate-order generator.  It contains none of the simulator's
arithmetic: no start/end times, makespans, bubbles or memory peaks.
"""
from .configs import CONFIGS, GIB_IN_UNITS, SegmentSpec, WorkloadConfig, get
from .instance import (KIND_B, KIND_F, Instance, Problem, comm_from_tokens,
                       compile_instance, make_instance, make_problem,
                       op_cost_from_tokens, pipeline_instance)
from .orders import (MODE_1F1B, MODE_LIST, OrderGenerator, build, generator_for,
                     gpipe_rank, one_f_one_b_rank, op_id, pack, unpack)

__all__ = [
    "CONFIGS", "GIB_IN_UNITS", "SegmentSpec", "WorkloadConfig", "get",
    "KIND_B", "KIND_F", "Instance", "Problem", "comm_from_tokens",
    "compile_instance", "make_instance", "make_problem", "op_cost_from_tokens",
    "pipeline_instance", "MODE_1F1B", "MODE_LIST", "OrderGenerator", "build",
    "generator_for", "gpipe_rank", "one_f_one_b_rank", "op_id", "pack", "unpack",
]
from .priorities import (expansion_draw, fifo_priorities, priority_groups,  # noqa: E402
                         rollout_priorities)

__all__ += ["expansion_draw", "fifo_priorities", "priority_groups", "rollout_priorities"]
