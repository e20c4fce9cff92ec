"""The C ABI from plain C: tests/c_consumer.c is built with gcc as C99
(-Wall -Wextra -Werror -pedantic) against include/infs.h, linked to
libinfs.so, and run without a GPU (dry-run context).  Its step count and
token totals must equal the oracle simulator's; its FPTAS grouping the
oracle's Algorithm 2."""

import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import fptas_assign, simulate
from paper_2506_22950_amd import infs

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LENGTHS = [5, 17, 3, 9, 12, 1, 30, 8, 8, 2]
PRED = [6.0, 15.5, 2.5, 11.0, 12.0, 1.5, 28.0, 7.0, 9.0, 2.0]
M, LAYERS = 4, 2


@pytest.fixture(scope="module")
def consumer(tmp_path_factory):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    lib_dir = os.path.dirname(infs.LIB_PATH)
    assert os.path.exists(infs.LIB_PATH), "build libinfs.so first"
    exe = str(tmp_path_factory.mktemp("c") / "c_consumer")
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-I" + os.path.join(ROOT, "include"),
           os.path.join(HERE, "c_consumer.c"), "-o", exe, "-L" + lib_dir, "-linfs", "-Wl,-rpath," + lib_dir]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return exe


def _run(exe, policy):
    r = subprocess.run([exe, str(policy)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    out = {}
    for ln in r.stdout.splitlines():
        k, _, v = ln.partition(" = ")
        out[k.strip()] = v.strip()
    return out


@pytest.mark.parametrize("policy", ["naive", "fifo", "sjf", "fptas_sjf"])
def test_c_consumer_matches_oracle(consumer, policy):
    out = _run(consumer, infs.POLICY[policy])
    sim = simulate(np.array(LENGTHS), M, policy, pred=np.array(PRED))
    assert int(out["steps"]) == sim.steps
    assert int(out["stats_steps"]) == sim.steps
    assert int(out["launches"]) == sim.steps * LAYERS
    assert int(out["tokens"]) == sum(LENGTHS)
    assert out["kernel"] == "bf16 0 head_dim 64 hpk 2 mfma 0 rows 8"
    assert int(out["decode_before_prefill"].split()[0]) == infs.E_STATE
    assert int(out["refill_live_slot"].split()[0]) == infs.E_STATE
    assert int(out["second_decode_same_layer"]) == infs.E_STATE
    assert int(out["retire_empty_slot"]) == infs.E_STATE
    group, pos = fptas_assign(np.array(PRED), M)
    assert [int(x) for x in out["fptas_group"].split()] == list(group)
    assert [int(x) for x in out["fptas_pos"].split()] == list(pos)
