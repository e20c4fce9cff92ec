"""The host runtime under AddressSanitizer and UndefinedBehaviorSanitizer.

runtime.cpp and sched.cpp are rebuilt with host-only sanitizers
(build.build_sanitized: every -fsanitize= applies to host code only) and the
host-side suites -- the C ABI from Python (test_abi_host.py), the dry-run
state machine (test_state_machine.py), the plain C consumer
(test_c_consumer.py) and the step-launch plan through the ABI
(test_step_plan.py) -- run again against that build in a child process with
the sanitizer runtime preloaded.  Any report (an out-of-bounds access, a use
after free, undefined behaviour) fails the run.  No GPU is used: these suites
run dry-run contexts.  Leak checking is off: the Python interpreter keeps its
own allocations to the end by design."""

import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.sanitize

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SUITES = ["tests/test_abi_host.py", "tests/test_state_machine.py", "tests/test_c_consumer.py",
          "tests/test_step_plan.py::test_step_split_plan_hand_cases"]


def test_host_runtime_under_asan_and_ubsan():
    from paper_2506_22950_amd import build

    lib = build.build_sanitized()
    env = dict(os.environ)
    env.update(INFS_LIBRARY=lib, LD_PRELOAD=build.sanitizer_runtime(),
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    env.pop("PYTEST_XDIST_WORKER", None)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-p", "no:xdist",
                        "-m", "not gpu", *SUITES], cwd=ROOT, env=env, capture_output=True, text=True, timeout=1200)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-6000:]
    assert r.returncode == 0, out[-6000:]
    assert " passed" in out
    print(out.strip().splitlines()[-1])
