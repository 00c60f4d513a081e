"""ambptt: backpropagation through time under asynchronous multistage
checkpointing on one AMD Instinct MI355X (gfx950).

The compute path is libambptt.so (HIP kernels, checkpoint tiers, executor,
schedule generator) behind the C ABI in include/ambptt.h; this package only
marshals torch tensors into it.
"""
from .api import (ProblemSpec, Runner, interval_from_timings, query, resident_program, revolve_advances, schedule_evals,
                  schedule_text, schedule_text_costs, schedule_text_online, schedule_text_sized, schedule_text_starts,
                  version)
from ._lib import AmbpttError, LIB_PATH, load

__all__ = ["ProblemSpec", "Runner", "interval_from_timings", "query", "resident_program", "revolve_advances", "schedule_evals", "schedule_text",
           "schedule_text_costs", "schedule_text_online", "schedule_text_sized", "schedule_text_starts", "version", "AmbpttError", "LIB_PATH", "load"]
