"""CPU oracle for shared-prefix continuous-sampling decode.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check in
``__graft_entry__`` and the CPU-baseline leg of ``bench.py`` may import or run
anything in this package.  The GPU library never calls it, and it shares no
code with the GPU library: the two meet only at the seeded input generator in
``workload/``.

Four parts, all plain and slow on purpose:

* ``attention`` -- float64 softmax attention of a decode query over the
  concatenation of the shared prompt KV and the sample's own response KV
  (Sections 2.1, 3.1 and 3.2 of the paper: one prompt KV cache shared by the
  whole group, one private response buffer per active sample).
* ``fp8`` -- OCP E4M3 rounding, for the FP8-stored KV cache (the paper's
  future-work direction of KV cache compression).
* ``simulator`` -- the step-by-step slot / refill process of naive micro
  sampling groups (Section 3.1), fixed-slot continuous sampling (Section 3.2)
  continuous refill in FIFO or shortest-job-first order (Algorithms 1
  and 3), FPTAS micro-group assignment (Algorithm 2) alone or followed by
  shortest-job-first refill, longest-first list scheduling, and
  dynamic-slot sampling from an unbounded stream (Section 3.2, mode 2).
* ``optimum`` -- the post-hoc optimum of Tables 1 and 2 ("Infinite*"): the
  fewest running steps of any assignment of the samples to the slots.

Every function is pinned by the ``-m "not gpu"`` tests against closed forms,
a library routine, brute force and a hand-derived worked example.
"""

from .attention import attend, attend_slot, attention_weights, default_scale
from .fp8 import E4M3_MAX, decode_e4m3, encode_e4m3, round_e4m3
from .optimum import brute_force as optimum_brute_force
from .optimum import lower_bound as optimum_lower_bound
from .optimum import makespan, optimum
from .simulator import (FPTAS_EPSILON, POLICIES, DynamicResult, SimResult, fptas_assign, simulate,
                        simulate_dynamic, simulate_group)

__all__ = [
    "E4M3_MAX",
    "decode_e4m3",
    "encode_e4m3",
    "round_e4m3",
    "attend",
    "attend_slot",
    "attention_weights",
    "default_scale",
    "FPTAS_EPSILON",
    "POLICIES",
    "fptas_assign",
    "SimResult",
    "DynamicResult",
    "simulate_dynamic",
    "simulate",
    "simulate_group",
    "optimum",
    "optimum_lower_bound",
    "optimum_brute_force",
    "makespan",
]
