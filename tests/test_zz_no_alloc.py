"""The allocation-free entry point infs_decode_step_static against infs_decode_step.

Both decode the same group with the same kernels; the static variant takes its
split-K workspace and arrival counters from the library's static device array
instead of the context's.  Two group decodes in a row, the second with a
smaller workspace (fewer slots and KV heads, so the array still holds the first
one's larger contents): step logs and token counters equal, every captured
output bitwise equal to the regular entry point's and within the bf16
tolerance of the float64 oracle.
"""

import numpy as np
import pytest

from paper_2506_22950_amd import infs
from tests.gpu_harness import check_against_oracle, oracle_log, run_gpu_group, say
from workload import Workload, get_config

pytestmark = pytest.mark.gpu


def _both(cfg, policy, split):
    wl = Workload(cfg)
    want = oracle_log(cfg, wl, policy)
    every = lambda k: k % 2 == 0 or k == len(want) - 1  # noqa: E731
    runs = {}
    for entry in ("decode_step", "decode_step_static"):
        say(f"  [{cfg.name} {entry}] G={cfg.samples_per_prompt} m={cfg.slots_per_prompt} Hkv={cfg.num_kv_heads}")
        _, log, steps, cap, tokens, _ = run_gpu_group(cfg, policy, wl=wl, split=split, capture=every, entry=entry)
        assert log == want and steps == len(want)
        assert np.array_equal(tokens, wl.L)
        runs[entry] = cap
    a, b = runs["decode_step"], runs["decode_step_static"]
    assert a.keys() == b.keys()
    for k in a:
        assert np.array_equal(a[k], b[k]), f"step {k}: static entry point differs from decode_step"
    worst, n = check_against_oracle(cfg, wl, want, b)
    say(f"  [{cfg.name}] static == decode_step on {len(b)} steps; {n} outputs vs oracle, max abs err {worst:.3g}")


def test_static_entry_point_two_groups_second_smaller():
    big = get_config("qwen3_1p7b_g64").with_(layers=2, prompt_lens=(700,), samples_per_prompt=40,
                                             length_dist=("lognormal", 4.5, 1.0, 1, 600), max_suffix_len=600,
                                             pool_rows=None)
    small = get_config("qwen3_1p7b_l1_g32").with_(num_q_heads=8, num_kv_heads=4, prompt_lens=(200,),
                                                  samples_per_prompt=10, slots_per_prompt=4,
                                                  length_dist=("lognormal", 3.5, 1.0, 1, 150), max_suffix_len=150)
    _both(big, "sjf", 128)
    _both(small, "fifo", 128)
