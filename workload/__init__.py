"""Seeded synthetic inputs for shared-prefix group decoding.

This package only draws inputs: completion lengths, predicted lengths and the
Q/K/V rows a decode step consumes.  It holds none of the attention or
scheduling arithmetic, so both the CPU oracle and the GPU harness can use it
without sharing any of the method's code.
"""

from .configs import CONFIGS, GroupConfig, get_config
from .gen import (SCHEDULER_STUDY, Workload, bf16_bits_to_f64, f32_to_bf16_bits, scheduler_study_lengths,
                  scheduler_study_stream, splitmix64)

__all__ = [
    "CONFIGS",
    "GroupConfig",
    "get_config",
    "SCHEDULER_STUDY",
    "Workload",
    "bf16_bits_to_f64",
    "f32_to_bf16_bits",
    "scheduler_study_lengths",
    "scheduler_study_stream",
    "splitmix64",
]
