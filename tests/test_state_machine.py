"""The host state machine of the C ABI (slots, steps, pages, prefill) against
a small reference model written from the header's contract, on long seeded
random call sequences in dry-run contexts (no GPU): every call's status, and
after it every slot's (sample, length) and the step / launch / token totals,
must agree.  Errors must leave the state unchanged."""

import numpy as np
import pytest

from paper_2506_22950_amd import infs
from paper_2506_22950_amd.group import context_for
from workload import get_config

PAGE = 16


class Model:
    def __init__(self, NP, m, G, L, P, cap, pages):
        self.NP, self.m, self.G, self.L, self.P, self.cap = NP, m, G, L, P, cap
        self.S = NP * m
        self.free = pages
        self.sample = [-1] * self.S
        self.len = [0] * self.S
        self.pages = [0] * self.S
        self.dispatched = [[False] * G for _ in range(NP)]
        self.plen = [-1] * NP
        self.prefilled = [[False] * L for _ in range(NP)]
        self.step_open = False
        self.done = [False] * L
        self.steps = self.launches = self.tokens = 0

    def live(self, p):
        return any(self.sample[s] >= 0 for s in range(p * self.m, (p + 1) * self.m))

    def refill(self, s, p, i):
        if not (0 <= s < self.S) or p != s // self.m or not (0 <= i < self.G):
            return infs.E_ARG
        if self.step_open or self.sample[s] >= 0:
            return infs.E_STATE
        if self.dispatched[p][i]:
            return infs.E_DUP
        self.dispatched[p][i] = True
        self.sample[s], self.len[s], self.pages[s] = i, 0, 0
        return infs.OK

    def retire(self, s):
        if not (0 <= s < self.S):
            return infs.E_ARG
        if self.step_open or self.sample[s] < 0:
            return infs.E_STATE
        self.free += self.pages[s]
        self.sample[s], self.len[s], self.pages[s] = -1, 0, 0
        return infs.OK

    def prefill(self, p, layer, n):
        if not (0 <= p < self.NP) or not (0 <= layer < self.L) or not (0 <= n <= self.P):
            return infs.E_ARG
        if self.plen[p] >= 0 and self.plen[p] != n:
            return infs.E_ARG
        if self.step_open:
            return infs.E_STATE
        self.plen[p] = n
        self.prefilled[p][layer] = True
        return infs.OK

    def decode(self, layer):
        if not (0 <= layer < self.L):
            return infs.E_ARG
        if self.step_open and self.done[layer]:
            return infs.E_STATE
        if any(self.live(p) and not self.prefilled[p][layer] for p in range(self.NP)):
            return infs.E_STATE
        if not self.step_open:
            live = [s for s in range(self.S) if self.sample[s] >= 0]
            if any(self.len[s] + 1 > self.cap for s in live):
                return infs.E_CAPACITY
            need = sum(1 for s in live if self.len[s] % PAGE == 0)
            if need > self.free:
                return infs.E_CAPACITY
            for s in live:
                if self.len[s] % PAGE == 0:
                    self.pages[s] += 1
            self.free -= need
            self.step_open = True
            self.done = [False] * self.L
        self.done[layer] = True
        self.launches += 1
        return infs.OK

    def end(self):
        if not self.step_open or not all(self.done):
            return infs.E_STATE
        for s in range(self.S):
            if self.sample[s] >= 0:
                self.len[s] += 1
                self.tokens += 1
        self.steps += 1
        self.step_open = False
        return infs.OK


def _status(fn, *a):
    try:
        fn(*a)
        return infs.OK
    except infs.InfsError as e:
        return e.status


@pytest.mark.parametrize("seed,NP,m,G,L,P,cap,pages", [
    (1, 1, 4, 8, 2, 32, 40, 0),
    (2, 2, 3, 5, 1, 40, 20, 4),      # a small page pool: exhaustion and recycling
    (3, 3, 2, 6, 3, 17, 33, 0),
    (4, 1, 8, 20, 1, 64, 18, 3),
])
def test_random_call_sequences(seed, NP, m, G, L, P, cap, pages):
    rng = np.random.default_rng(seed)
    cfg = get_config("tiny_f32").with_(layers=L, prompt_lens=(P,) * NP, samples_per_prompt=G, slots_per_prompt=m,
                                       max_suffix_len=cap)
    ctx = context_for(cfg, dry_run=True, num_pages=pages)
    S = NP * m
    model = Model(NP, m, G, L, P, cap, pages if pages else S * -(-cap // PAGE))
    none4 = (None, None, None, None)
    counts = {}
    for k in range(4000):
        if k % 500 == 499:  # infs_reset: a fresh group
            ctx.reset()
            model = Model(NP, m, G, L, P, cap, pages if pages else S * -(-cap // PAGE))
            continue
        op = rng.choice(["refill", "retire", "prefill", "decode", "end", "step"], p=[.25, .1, .1, .1, .05, .4])
        if op == "refill":
            empty = [x for x in range(S) if model.sample[x] < 0]
            s = int(rng.choice(empty)) if empty and rng.random() < 0.8 else int(rng.integers(-1, S + 1))
            p = s // m if rng.random() < 0.9 else int(rng.integers(0, NP + 1))
            pp = min(max(p, 0), NP - 1)
            fresh = [i for i in range(G) if not model.dispatched[pp][i]]
            i = int(rng.choice(fresh)) if fresh and rng.random() < 0.8 else int(rng.integers(-1, G + 1))
            got, want = _status(ctx.refill_slot, s, p, i), model.refill(s, p, i)
        elif op == "retire":
            live = [x for x in range(S) if model.sample[x] >= 0]
            s = int(rng.choice(live)) if live and rng.random() < 0.8 else int(rng.integers(-1, S + 1))
            got, want = _status(ctx.retire_slot, s), model.retire(s)
        elif op == "prefill":
            valid = rng.random() < 0.8
            p = int(rng.integers(0, NP)) if valid else int(rng.integers(-1, NP + 1))
            layer = int(rng.integers(0, L)) if valid else int(rng.integers(-1, L + 1))
            n = P if valid else int(rng.integers(-1, P + 2))
            got, want = _status(ctx.prefill_shared, p, layer, n, None, None), model.prefill(p, layer, n)
        elif op == "decode":
            layer = int(rng.integers(-1, L + 1))
            got, want = _status(ctx.decode_step, layer, *none4), model.decode(layer)
        elif op == "end":
            got, want = _status(ctx.end_step), model.end()
        else:  # a whole step: every layer, then end (or the first error)
            got = want = infs.OK
            for layer in range(L):
                got, want = _status(ctx.decode_step, layer, *none4), model.decode(layer)
                if got != want or got != infs.OK:
                    break
            if got == want == infs.OK:
                got, want = _status(ctx.end_step), model.end()
        assert got == want, (op, got, want)
        counts[want] = counts.get(want, 0) + 1
        for s in range(S):
            assert ctx.slot_state(s) == (model.sample[s], model.len[s]), s
        st = ctx.get_stats()
        assert (st.steps, st.launches, st.tokens) == (model.steps, model.launches, model.tokens)
    ctx.destroy()
    # every outcome was exercised
    for code in (infs.OK, infs.E_ARG, infs.E_STATE, infs.E_DUP):
        assert counts.get(code, 0) > 0, (code, counts)
