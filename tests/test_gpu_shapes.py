"""GPU parity of every decode kernel instantiation (the table in
tests/shape_table.py) on a small workload that selects it: one layer, a
70-token prompt, m slots refilled FIFO, every other step compared with the
float64 oracle (bf16 and the E4M3 cache within 1e-2 against the oracle on the
stored values, fp32 within 1e-5); step log and token counters bit-exact."""

import numpy as np
import pytest

from tests.gpu_harness import check_against_oracle, oracle_log, run_gpu_group, say
from tests.shape_table import ENTRIES, case_for, case_id
from workload import Workload

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("entry", ENTRIES, ids=case_id)
def test_instantiation_parity(entry):
    cfg, probe_k, want = case_for(entry)
    kv8 = entry[5]
    wl = Workload(cfg)
    want_log = oracle_log(cfg, wl, "fifo", reuse=probe_k)
    info = {}

    def inspect(ctx, step, log):
        if not info:
            info.update(ctx.kernel_info())

    probe = {} if probe_k else None
    _, log, steps, captured, tokens, _ = run_gpu_group(cfg, "fifo", wl=wl, reuse=probe_k, probe=probe,
                                                       kv_fp8=kv8, inspect=inspect,
                                                       capture=lambda k: k % 2 == 0 or k == len(want_log) - 1)
    for k, v in want.items():
        assert info[k] == v, (k, info)
    assert log == want_log and steps == len(want_log)
    assert np.array_equal(tokens, wl.L)
    worst, n = check_against_oracle(cfg, wl, log, captured, kv_fp8=kv8)
    if probe_k:
        wp, npr = check_against_oracle(cfg, wl, probe["log"], probe["captured"], kv_fp8=kv8)
        worst, n = max(worst, wp), n + npr
    say(f"  [{cfg.name}] {n} outputs, max abs err {worst:.3g}")
