"""Pins for the post-hoc optimum ("Infinite*", Table 1 caption and Section 5.4).

The oracle decides the smallest slot capacity that holds all samples; these
checks tie it to things it does not compute itself: the definition by brute
force over every assignment, hand-worked instances (among them the worked
example's 8 and the classic cases where longest-first list scheduling is not
optimal), closed forms for m = 1 and m >= G, and the bounds that any
schedule obeys.  The library's branch and bound (infs_sched_optimum) is then
checked against the oracle.
"""

import json
import os

import numpy as np
import pytest

from oracle import makespan, optimum, optimum_brute_force, optimum_lower_bound, simulate

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "sim_worked_example.json")


def test_worked_example():
    # G=6, m=2, L=[3,1,4,1,5,2]: {3,5} against {1,4,1,2} takes 8 steps, and
    # sum/m = 8 shows that nothing is shorter.
    g = json.load(open(GOLDEN))
    val, slot = optimum(g["L"], g["m"])
    assert val == g["optimum_makespan"] == 8
    assert makespan(g["L"], slot, g["m"]) == 8


@pytest.mark.parametrize("L,m,opt,lpt", [
    # Hand-worked.  Longest-first list scheduling (LPT) puts 3,3 apart, then
    # 2,2 on top, then the last 2 on either side (7); the optimum is 3+3 | 2+2+2.
    ([3, 3, 2, 2, 2], 2, 6, 7),
    # Graham's tight case for m = 3: 5,5,4,4,3,3,3.  LPT: 5 | 5 | 4, then 4 on
    # the third slot (8), 3 on the first two (8, 8), the last 3 on top (11);
    # the optimum is 5+4 | 5+4 | 3+3+3 = 9.
    ([5, 5, 4, 4, 3, 3, 3], 3, 9, 11),
    # One long sample dominates: it alone sets the steps.
    ([10, 1, 1, 1], 2, 10, 10),
    # Perfect split of 1..8 (sum 36) into 4 slots of 9: 8+1, 7+2, 6+3, 5+4.
    ([1, 2, 3, 4, 5, 6, 7, 8], 4, 9, 9),
])
def test_hand_cases(L, m, opt, lpt):
    val, slot = optimum(L, m)
    assert val == opt and makespan(L, slot, m) == opt
    assert simulate(L, m, "lpt", pred=L).steps == lpt


def test_brute_force_random():
    rng = np.random.default_rng(11)
    for _ in range(400):
        G = int(rng.integers(1, 9))
        m = int(rng.integers(1, 5))
        L = rng.integers(1, 20, size=G)
        val, slot = optimum(L, m)
        assert val == optimum_brute_force(L, m), (L, m)
        assert makespan(L, slot, m) == val


def test_closed_forms_and_bounds():
    rng = np.random.default_rng(12)
    for _ in range(200):
        G = int(rng.integers(1, 14))
        m = int(rng.integers(1, 6))
        L = rng.integers(1, 50, size=G)
        val, slot = optimum(L, m)
        if m == 1:
            assert val == L.sum()
        if m >= G:
            assert val == L.max()
        lb = optimum_lower_bound(L, m)
        assert lb == max(-(-int(L.sum()) // m), int(L.max()))
        assert lb <= val
        # every online policy is a schedule too, so none beats the optimum
        for policy in ("fifo", "sjf", "lpt", "fixed_row", "naive"):
            assert simulate(L, m, policy, pred=L).steps >= val
        # Graham: LPT is within 4/3 - 1/(3m) of the optimum
        assert simulate(L, m, "lpt", pred=L).steps <= (4 / 3 - 1 / (3 * m)) * val + 1e-9


def test_budget_reports_unsolved():
    # A budget of one node cannot decide a tight instance.
    val, slot = optimum([7, 6, 5, 4, 3, 3, 2, 2, 1], 3, max_nodes=1)
    assert val is None and slot is None
