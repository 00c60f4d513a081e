"""Seeded synthetic workloads for long-sequence BPTT.

This module is shared by the CPU oracle (tests, CPU baseline) and the GPU
path (tests, bench).  It holds workload shapes and the seeded generators of
their inputs, and none of the method's arithmetic: no cell update, no adjoint,
no schedule.

The paper measures on a numpy LSTM for text generation (Section 5) whose code
and data are not available; the workloads here stand in for it as synthetic
recurrent problems of the long-sequence shape the paper targets (hundreds to
tens of thousands of steps, uniform state size per step).

Every array is drawn from numpy's PCG64 stream seeded by a SeedSequence of
(base seed, stream id, index), so that any time slice ``x[t0:t1]`` or any
layer's weights can be regenerated on its own, in any order, with the same
values.
"""
from .workloads import (Workload, WORKLOADS, get, x_slice, params, layer_params, initial_state,
                        f32_to_bf16_bits, bf16_bits_to_f32)

__all__ = ["Workload", "WORKLOADS", "get", "x_slice", "params", "layer_params", "initial_state",
           "f32_to_bf16_bits", "bf16_bits_to_f32"]
