"""The post-hoc optimum of a group decode ("Infinite*").

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper's reference schedule in Tables 1 and 2 places every response after
generation, when all lengths are known, so that the group needs the fewest
running steps possible (Table 1 caption; Section 5.4).  A slot runs the
samples it is given back to back -- a freed slot's next sample decodes at the
following step, with no idle step between -- so a slot holding the sample set
A is busy for sum(L_i, i in A) steps, and any split of the samples into m sets
can be run that way.  The optimum is therefore

    OPT = min over partitions of the G samples into m sets of the largest set sum,

the makespan problem P||Cmax.  Written here as the smallest capacity C at
which the samples can be packed into m slots: C runs upward from the simple
lower bound max(ceil(sum/m), max L), and each C is decided by a depth-first
search that places the samples, longest first, into slots of capacity C.
Slots whose current loads are equal are interchangeable, so only the first
of them is tried, and a search state (next sample, multiset of slot loads)
that failed is remembered.  The search is exact; a node budget makes it report
"unsolved" rather than run for long on a hard instance.
"""

import math
from typing import List, Optional, Sequence, Tuple


def lower_bound(L: Sequence[int], m: int) -> int:
    """max(ceil(sum L / m), max L): no schedule of m slots is shorter."""
    L = [int(x) for x in L]
    return max(-(-sum(L) // m), max(L))


def _fits(sizes: List[int], m: int, cap: int, budget: List[int]) -> Optional[List[int]]:
    """A slot for every size (sizes in descending order) with no slot above
    `cap`, or None if there is none.  budget[0] counts down the search nodes;
    at zero the search stops and raises _OutOfBudget.

    Two rules cut the search without losing a packing:
    * free capacity that no remaining sample fits into (it is smaller than the
      smallest one) stays empty; once that waste exceeds the slack
      m * cap - sum(sizes), no packing completes;
    * a sample that fills a slot exactly is put there and nowhere else (any
      packing that puts it elsewhere can swap it with that slot's remaining
      contents).
    Slots are tried emptiest first (equal loads once).  Whether the samples
    from i on can still be placed depends only on i and the multiset of slot
    loads, so a (i, sorted loads) state that failed once is not searched
    again."""
    n = len(sizes)
    loads = [0] * m
    where = [0] * n
    slack = m * cap - sum(sizes)
    if slack < 0:
        return None
    failed = set()

    def place(i: int) -> bool:
        if i == n:
            return True
        budget[0] -= 1
        if budget[0] < 0:
            raise _OutOfBudget
        state = (i, tuple(sorted(loads)))
        if state in failed:
            return False
        if not _try(i):
            failed.add(state)
            return False
        return True

    def _try(i: int) -> bool:
        smallest = sizes[-1]
        waste = sum(cap - x for x in loads if cap - x < smallest)
        if waste > slack:
            return False
        x = sizes[i]
        exact = [s for s in range(m) if loads[s] + x == cap]
        if exact:
            candidates = exact[:1]
        else:
            candidates, seen = [], set()
            for s in sorted(range(m), key=lambda s: (loads[s], s)):
                if loads[s] + x <= cap and loads[s] not in seen:
                    seen.add(loads[s])
                    candidates.append(s)
        for s in candidates:
            loads[s] += x
            where[i] = s
            if place(i + 1):
                return True
            loads[s] -= x
        return False

    return list(where) if place(0) else None


class _OutOfBudget(Exception):
    pass


def optimum(L: Sequence[int], m: int, max_nodes: int = 2_000_000) -> Tuple[Optional[int], Optional[List[int]]]:
    """(OPT, slot of each sample) for true lengths L on m slots, or
    (None, None) when the node budget ran out before the answer was proven."""
    L = [int(x) for x in L]
    if m < 1 or not L or min(L) < 1:
        raise ValueError("need m >= 1 and at least one sample, each with >= 1 token")
    order = sorted(range(len(L)), key=lambda i: (-L[i], i))
    sizes = [L[i] for i in order]
    budget = [max_nodes]
    cap = lower_bound(L, m)
    total = sum(L)
    while cap <= total:
        try:
            where = _fits(sizes, m, cap, budget)
        except _OutOfBudget:
            return None, None
        if where is not None:
            slot = [0] * len(L)
            for k, i in enumerate(order):
                slot[i] = where[k]
            return cap, slot
        cap += 1
    raise AssertionError("unreachable: every sample fits one slot of capacity sum(L)")


def makespan(L: Sequence[int], slot: Sequence[int], m: int) -> int:
    """Running steps of the post-hoc schedule that gives sample i to slot[i]."""
    loads = [0] * m
    for x, s in zip(L, slot):
        loads[s] += int(x)
    return max(loads)


def brute_force(L: Sequence[int], m: int) -> int:
    """The definition itself, over all m^G assignments (tiny G only)."""
    import itertools

    L = [int(x) for x in L]
    best = math.inf
    for assign in itertools.product(range(m), repeat=len(L)):
        best = min(best, makespan(L, assign, m))
    return int(best)
