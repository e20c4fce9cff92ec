"""Step-by-step slot / refill simulator.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The process follows the paper's decode loop (Algorithm 1, phase 2): at every
running step each active slot decodes one token of its sample (a running step
is one token-generation round over the g slots, Section 5.1); a sample that
has produced its last token releases its slot, and the slot receives the next
sample, which decodes its first token at the following step (Section 3.2).

Refill policies:

* ``naive``     -- micro sampling groups decoded one after another
                   (Section 3.1): slots are refilled only once every slot is
                   empty, with the next m sample ids in order.
* ``fixed_row`` -- fixed-slot continuous sampling (Section 3.2, mode 1): slot
                   s runs samples s, s+m, s+2m, ... back to back.
* ``fifo``      -- continuous refill from the pending pool, lowest sample id
                   first.
* ``sjf``       -- shortest-job-first refill (Algorithm 3): the pending sample
                   with the smallest predicted length, ties to the lowest id.
* ``fptas``     -- static pre-planning only (Table 2's "FPTAS only"): the
                   samples are grouped into m bins by Algorithm 2 on the
                   predicted lengths, and slot s runs bin s in position order.
* ``fptas_sjf`` -- the two-stage scheduler of Algorithm 1 (Table 2's
                   "Infinite"): every slot starts with position 0 of its bin,
                   and every later refill is shortest-job-first.
* ``lpt``       -- continuous refill, longest predicted length first, ties to
                   the lowest id.  Given the true lengths this is a post-hoc
                   list schedule: an upper bound on the post-hoc optimum of
                   Tables 1 and 2 ("Infinite*", ``optimum.optimum``), within
                   4/3 - 1/(3m) of it (Graham 1969).

Readings where the paper is silent: a sample of length L holds its slot for
exactly L steps; when several slots free up in one step they are refilled in
ascending slot order; the initial fill uses the same policy as every refill
(for ``fptas_sjf``: position 0 of the slot's bin, or shortest-job-first if
the bin is empty or its first sample already left); Algorithm 3's candidate
set is the samples neither finished nor already dispatched (its ``mask`` being
the runtime dispatch record); Algorithm 2 runs with one bin per slot.
"""

import math

from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import numpy as np

POLICIES = ("naive", "fixed_row", "fifo", "sjf", "fptas", "fptas_sjf", "lpt")
NEEDS_PRED = ("sjf", "fptas", "fptas_sjf", "lpt")
FPTAS_EPSILON = 0.1


def fptas_assign(pred, N: int, eps: float = FPTAS_EPSILON):
    """Algorithm 2 (FPTAS-based micro group assignment), step by step.

    The predicted lengths are scaled by K = eps * S / N (S their sum) and
    rounded up to integers; the bin capacity is the rounded-up mean of the
    scaled sizes over the N bins; samples are taken in descending scaled
    size (ties: lower id first) and each goes to the first bin it fits in.
    The paper leaves unplaced samples unspecified: such a sample goes to the
    bin with the smallest scaled load (lowest index on ties).

    Returns (group, pos): sample i is the pos[i]-th sample of bin group[i].
    Floating point: S is summed in id order and K = (eps * S) / N, in float64.
    """
    pred = [float(x) for x in pred]
    G = len(pred)
    if N < 1:
        raise ValueError("N must be >= 1")
    S = 0.0
    for x in pred:
        S += x
    K = (eps * S) / N
    if not (K > 0.0):
        raise ValueError("the predicted lengths must have a positive sum")
    size = [int(math.ceil(x / K)) for x in pred]
    cap = -(-sum(size) // N)  # ceil of the integer mean
    load = [0] * N
    members = [[] for _ in range(N)]
    group = [-1] * G
    pos = [-1] * G
    for i in sorted(range(G), key=lambda i: (-size[i], i)):
        target = None
        for n in range(N):
            if load[n] + size[i] <= cap:
                target = n
                break
        if target is None:
            target = min(range(N), key=lambda n: (load[n], n))
        group[i] = target
        pos[i] = len(members[target])
        members[target].append(i)
        load[target] += size[i]
    return group, pos


@dataclass
class SimResult:
    steps: int
    # log[k][s] = (sample, t) for slot s at step k+1 (t = tokens after this step), or None
    log: List[Tuple[Optional[Tuple[int, int]], ...]]
    tokens: np.ndarray                       # tokens decoded per sample
    dispatch: List[Tuple[int, int, int]]     # (steps completed before, slot, sample)
    finish_step: np.ndarray                  # step at which each sample produced its last token


def simulate(L, m: int, policy: str, pred=None, reuse: int = 0) -> SimResult:
    """Simulate one prompt's group of G = len(L) samples on m slots.

    reuse = k > 0: prefix reuse (Section 4).  Every sample has already decoded
    min(L_i, k) probe tokens before the first step; a dispatched sample
    resumes at token k+1 and holds its slot for L_i - k steps, and a sample
    with L_i <= k finished in the probe phase: when the policy picks it, it is
    counted as finished at once and the slot asks the policy again.  Log
    entries carry the response length including the probe tokens.
    """
    L = [int(x) for x in L]
    G = len(L)
    if m < 1:
        raise ValueError("m must be >= 1")
    if any(x < 1 for x in L):
        raise ValueError("every sample has at least one token")
    if policy not in POLICIES:
        raise ValueError(f"unknown policy {policy!r}")
    if reuse < 0:
        raise ValueError("reuse must be >= 0")
    if policy in NEEDS_PRED:
        if pred is None:
            raise ValueError(f"{policy} needs predicted lengths")
        pred = [float(x) for x in pred]
    bins = None
    if policy in ("fptas", "fptas_sjf"):
        group, pos = fptas_assign(pred, m)
        bins = [[] for _ in range(m)]
        for i in sorted(range(G), key=lambda i: (group[i], pos[i])):
            bins[group[i]].append(i)
    bin_next = [0] * m            # fptas: next position of each slot's bin
    started = [False] * m         # fptas_sjf: slot has had its initial fill

    slot_sample = [None] * m      # sample id held by each slot, or None
    slot_len = [0] * m            # tokens of that sample so far (probe tokens included)
    pending = set(range(G))       # not yet dispatched
    row_next = list(range(m))     # fixed_row: next sample id of each slot
    naive = {"next": 0, "left": 0}  # naive: next id, ids left in the open micro group
    tokens = np.zeros(G, dtype=np.int64)
    finish = np.full(G, -1, dtype=np.int64)
    log = []
    dispatch = []
    step = 0

    def pick(s):
        """The policy's next sample for empty slot s, or None."""
        if policy == "naive":
            if naive["left"] == 0 and all(x is None for x in slot_sample) and naive["next"] < G:
                naive["left"] = min(m, G - naive["next"])
            if naive["left"] == 0:
                return None
            j = naive["next"]
            naive["next"] += 1
            naive["left"] -= 1
            return j
        if policy == "fixed_row":
            j = row_next[s]
            if j >= G:
                return None
            row_next[s] = j + m
            return j
        if policy == "fptas":
            if bin_next[s] >= len(bins[s]):
                return None
            j = bins[s][bin_next[s]]
            bin_next[s] += 1
            return j
        if not pending:
            return None
        if policy == "fifo":
            return min(pending)
        if policy == "lpt":
            return min(pending, key=lambda i: (-pred[i], i))
        if policy == "fptas_sjf" and not started[s]:
            started[s] = True
            if bins[s] and bins[s][0] in pending:
                return bins[s][0]
        return min(pending, key=lambda i: (pred[i], i))

    def fill():
        for s in range(m):
            while slot_sample[s] is None:
                j = pick(s)
                if j is None:
                    break
                pending.discard(j)
                dispatch.append((step, s, j))
                pre = min(L[j], reuse)
                tokens[j] = pre
                if pre == L[j]:          # finished within its probe tokens
                    finish[j] = step
                    continue
                slot_sample[s] = j
                slot_len[s] = pre

    fill()
    while any(x is not None for x in slot_sample):
        step += 1
        row = []
        for s in range(m):
            j = slot_sample[s]
            if j is None:
                row.append(None)
                continue
            slot_len[s] += 1
            tokens[j] += 1
            row.append((j, slot_len[s]))
        log.append(tuple(row))
        for s in range(m):
            j = slot_sample[s]
            if j is not None and slot_len[s] == L[j]:
                finish[j] = step
                slot_sample[s] = None
        fill()
    return SimResult(steps=step, log=log, tokens=tokens, dispatch=dispatch, finish_step=finish)


def simulate_group(L, m: int, policy: str, pred=None, reuse: int = 0):
    """Several prompts decoded in one batch, each with its own m slots and
    pending pool.  A step advances every prompt; the batch ends when the last
    prompt's group is done.  Returns (total steps, per-prompt SimResults)."""
    L = np.asarray(L)
    if L.ndim == 1:
        L = L[None, :]
    if pred is not None:
        pred = np.asarray(pred).reshape(L.shape)
    res = [simulate(L[p], m, policy, None if pred is None else pred[p], reuse) for p in range(L.shape[0])]
    return max(r.steps for r in res), res


@dataclass
class DynamicResult:
    steps: int
    log: List[Tuple[Optional[Tuple[int, int]], ...]]   # as SimResult.log
    accepted: List[int]                                 # the first `target` samples to complete
    mean_length: float                                  # their mean length (Table 1's length bias)


def simulate_dynamic(L_stream, m: int, target: int) -> DynamicResult:
    """Dynamic-slot continuous sampling (Section 3.2, mode 2).

    Samples come from an unbounded stream (ids 0, 1, 2, ... with lengths
    L_stream); a freed slot takes the next id at once, whatever the group
    structure.  Decoding stops at the end of the step in which the
    `target`-th sample completes; samples still decoding are discarded.
    Readings: completions within one step are counted in ascending slot
    order, and the stream must be long enough to reach `target` completions.
    """
    L = [int(x) for x in L_stream]
    if m < 1 or target < 1:
        raise ValueError("m and target must be >= 1")
    if any(x < 1 for x in L):
        raise ValueError("every sample has at least one token")
    slot_sample = [None] * m
    slot_len = [0] * m
    nxt = 0
    accepted = []
    log = []
    step = 0

    def fill():
        nonlocal nxt
        for s in range(m):
            if slot_sample[s] is None and nxt < len(L):
                slot_sample[s] = nxt
                slot_len[s] = 0
                nxt += 1

    fill()
    while len(accepted) < target:
        if all(x is None for x in slot_sample):
            raise ValueError("the stream ran out before the target number of completions")
        step += 1
        row = []
        for s in range(m):
            j = slot_sample[s]
            if j is None:
                row.append(None)
                continue
            slot_len[s] += 1
            row.append((j, slot_len[s]))
        log.append(tuple(row))
        for s in range(m):
            j = slot_sample[s]
            if j is not None and slot_len[s] == L[j]:
                if len(accepted) < target:
                    accepted.append(j)
                slot_sample[s] = None
        if len(accepted) < target:
            fill()
    return DynamicResult(steps=step, log=log, accepted=accepted,
                         mean_length=sum(L[i] for i in accepted) / len(accepted))
