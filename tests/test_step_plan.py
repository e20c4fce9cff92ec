"""The step launch's work split (csrc/step_plan.h) on the host:
tests/step_plan_check.cpp is built with g++ against the header alone and
checks, over random slot lengths and launch shapes, that the roles add up,
that the pieces of every live response are whole page ranges that tile it
(per wavefront too, as the kernel cuts them) within the bounds on pieces per
slot and pages per wavefront, that the cut matches an exhaustive search
for the smallest largest piece, and that longer prefix chunks are chosen
exactly when the per-layer chunks would give some producer two items."""

import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "paper_2506_22950_amd", "csrc")


@pytest.mark.parametrize("sanitize", [False, True], ids=["plain", "asan_ubsan"])
def test_step_plan_host_check(tmp_path, sanitize):
    # Also built with AddressSanitizer and UndefinedBehaviorSanitizer (g++, host code only):
    # any out-of-bounds access or undefined behaviour in the planner fails the run.
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path / "step_plan_check")
    flags = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all"] if sanitize else ["-O2"]
    r = subprocess.run(["g++", "-std=c++17", *flags, "-Wall", "-Wextra", "-Werror", "-I" + CSRC,
                        os.path.join(HERE, "step_plan_check.cpp"), "-o", exe], capture_output=True, text=True)
    if sanitize and r.returncode != 0 and "asan" in r.stderr.lower():
        pytest.skip("g++ sanitizer runtime not available")
    assert r.returncode == 0, r.stderr
    r = subprocess.run([exe, "20000"], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "failures 0" in r.stdout


def test_step_split_plan_hand_cases():
    # Through the C ABI, cases worked out by hand for the benchmark's launch shape (64 work-groups
    # per KV head, 16 slots: 4 merge work-groups, 60 producers; 16 prefix chunks of 128 tokens).
    from paper_2506_22950_amd import infs
    # 16 responses of 300 tokens: 32 chunks of 256 tokens; the chunk plan gives
    # min(16, 60 * 16 // 48) = 16 prefix and 44 response work-groups, which take one chunk
    # each, so the chunks stay.
    roles, pieces = infs.step_split_plan(64, [300] * 16, 16, 128, 256, 16)
    assert roles == dict(n_pre=16, n_suf=44, n_merge=4, items=32, cut=0)
    assert list(pieces) == [2] * 16
    # 16 responses of 1000 tokens (63 pages): 64 chunks for the chunk plan's 48 response
    # work-groups (60 * 16 // 80 = 12 prefix).  One prefix chunk each leaves 44 work-groups:
    # 2 pieces per slot (3 would need 48), largest 32 pages = 512 tokens, against a doubled
    # prefix weight of 256; two chunks per prefix work-group (8 of them) cost 2 * 256 = 512,
    # no better, so 16 prefix work-groups and 32 pieces.
    roles, pieces = infs.step_split_plan(64, [1000] * 16, 16, 128, 256, 16)
    assert roles == dict(n_pre=16, n_suf=44, n_merge=4, items=32, cut=1)
    assert list(pieces) == [2] * 16
    # mode 0 keeps the chunks and the proportional split
    roles, pieces = infs.step_split_plan(64, [1000] * 16, 16, 128, 256, 16, mode=0)
    assert roles == dict(n_pre=12, n_suf=48, n_merge=4, items=64, cut=0)
    # idle slots take nothing; arguments are checked
    roles, pieces = infs.step_split_plan(64, [0, 5, 0, 40], 2, 128, 256, 16)
    assert list(pieces) == [0, 1, 0, 1] and roles["items"] == 2
    with pytest.raises(infs.InfsError):
        infs.step_split_plan(64, [5000], 1, 128, 256, 16)   # longer than scmax * split
    with pytest.raises(infs.InfsError):
        infs.step_split_plan(1, [5], 1, 128, 256, 16)
