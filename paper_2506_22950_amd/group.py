"""Group decode through the C ABI: the runtime loop of Algorithm 1, phase 2.

Every running step decodes one token for each live slot through every layer
(``decode_step`` per layer, then ``end_step``); a sample that has produced its
last token releases its slot (``retire_slot``) and the refill policy of its
prompt hands the slot a pending sample (``refill_slot``), which decodes from the
next step on.  The host knows each sample's length (synthetic workloads), so it
never waits on the GPU inside the loop.
"""

from typing import Callable, List, Optional, Sequence

from . import infs


def context_for(cfg, stream=None, dry_run=False, split_tokens=0, num_pages=0, probe_tokens=0,
                kv_fp8=False, scale=0.0) -> infs.Context:
    """Create a context for a workload preset (workload.GroupConfig or alike);
    scale 0 is the default softmax scale 1/sqrt(head_dim)."""
    c = infs.make_config(
        num_layers=cfg.layers, num_q_heads=cfg.num_q_heads, num_kv_heads=cfg.num_kv_heads,
        head_dim=cfg.head_dim, num_prompts=cfg.num_prompts, slots_per_prompt=cfg.slots_per_prompt,
        samples_per_prompt=cfg.samples_per_prompt, max_prompt_len=max(cfg.prompt_lens),
        max_suffix_len=cfg.max_suffix_len, page_tokens=0, num_pages=num_pages,
        split_tokens=split_tokens, dtype=infs.BF16 if cfg.dtype == "bf16" else infs.F32,
        scale=scale, flags=(infs.FLAG_DRY_RUN if dry_run else 0) | (infs.FLAG_KV_FP8 if kv_fp8 else 0),
        probe_tokens=probe_tokens)
    return infs.Context(c, stream=None if dry_run else stream)


def schedulers_for(cfg, policy: str, pred=None) -> List[infs.Sched]:
    """One host scheduler per prompt."""
    out = []
    for p in range(cfg.num_prompts):
        out.append(infs.Sched(cfg.samples_per_prompt, cfg.slots_per_prompt, policy,
                              None if pred is None else pred[p]))
    return out


def probe_group(ctx: infs.Context, lengths, k: int, num_layers: int, provide: Callable,
                log: Optional[list] = None, after_step: Optional[Callable] = None, entry: str = "probe_step") -> int:
    """Probe phase of prefix reuse (Section 4): every sample decodes its first
    min(L_i, k) tokens against the shared prompt, in batches of up to
    ctx.probe_batch samples of one prompt; samples that finish within their
    probe tokens are released.  Returns the number of probe steps.

    provide(step, prompt, first, n, layer) -> (q, k_new, v_new, o) device
    buffers of that batch ([n, Hq, d], [n, Hkv, d], [n, Hkv, d], [n, Hq, d]).
    log, if given, receives one row per probe step: per batch position
    (prompt, sample, t) with t the probe length after this step, or None.
    after_step(step) is called after each end_probe_step.
    entry: "probe_step" (one launch per layer) or "probe_step_layers" (every
    layer of a probe step in one launch; the layer strides are read off the
    pointers provide returns for layers 0 and 1).
    """
    nb = ctx.probe_batch
    steps = 0
    for t in range(1, k + 1):
        for p, row in enumerate(lengths):
            G = len(row)
            for first in range(0, G, nb):
                n = min(nb, G - first)
                live = [int(row[first + j]) >= t for j in range(n)]
                if not any(live):
                    continue
                if entry == "probe_step_layers":
                    b0 = provide(steps, p, first, n, 0)
                    strides = [0, 0, 0]
                    if num_layers > 1 and b0[0] is not None:  # dry-run contexts take no buffers
                        b1 = provide(steps, p, first, n, 1)
                        strides = [b1[0] - b0[0], b1[1] - b0[1], b1[3] - b0[3]]
                        if b1[2] - b0[2] != strides[1]:
                            raise ValueError("k_new and v_new need the same layer stride")
                    ctx.probe_step_layers(p, first, n, live, *b0, *strides)
                else:
                    for layer in range(num_layers):
                        ctx.probe_step(layer, p, first, n, live, *provide(steps, p, first, n, layer))
                ctx.end_probe_step()
                if after_step is not None:
                    after_step(steps)
                if log is not None:
                    log.append(tuple((p, first + j, t) if live[j] else None for j in range(n)))
                steps += 1
    for p, row in enumerate(lengths):
        for i, x in enumerate(row):
            if int(x) <= k:
                ctx.release_sample(p, i)
    return steps


def decode_group(ctx: infs.Context, scheds: Sequence[infs.Sched], lengths, num_layers: int,
                 provide: Callable, after_step: Optional[Callable] = None,
                 log: Optional[list] = None, stop_after: Optional[int] = None,
                 accepted: Optional[list] = None, reuse: int = 0, entry: str = "decode_step") -> int:
    """Decode every sample of every prompt; returns the number of running steps.

    lengths[p][i]: true length of sample i of prompt p.
    provide(step, layer) -> (q, k_new, v_new, o) device buffers for that layer-step.
    after_step(step) is called after each end_step.
    log, if given, receives one tuple per step: for each slot (prompt, sample, t)
    with t the response length after this step, or None for an idle slot.
    stop_after: dynamic-slot sampling (Section 3.2, mode 2) -- the samples of a
    prompt form a stream, and once `stop_after` of them have completed (counted
    in ascending slot order within a step) the prompt stops: its samples still
    decoding are discarded (their slots retired) and it is not refilled.
    accepted, if given, receives per prompt the completed sample ids in order.
    reuse = k: the samples went through a probe phase of k tokens (probe_group);
    a dispatched sample resumes at token k+1, and one that finished within its
    probe tokens is skipped (the scheduler is told it is done at once).
    entry: the C call that decodes a layer -- "decode_step", or
    "decode_step_static" (split-K workspace in the library's static scratch) --
    or "decode_step_layers": every layer of a step in one launch, fed with the
    pointers provide(step, 0) returns, whose layers must be laid out densely
    ([L, S, H, d] for Q, the new K/V rows and O).  A function of the step
    number picks the entry step by step.
    """
    entries = {"decode_step": ctx.decode_step, "decode_step_static": ctx.decode_step_static,
               "decode_step_layers": None}
    entry_of = entry if callable(entry) else (lambda step: entry)
    NP = len(scheds)
    m = ctx.config.slots_per_prompt
    S = NP * m
    slot_sample = [-1] * S
    slot_len = [0] * S
    Ls = [[int(x) for x in row] for row in lengths]
    done = [[] for _ in range(NP)]
    stopped = [False] * NP

    def fill():
        for p in range(NP):
            if stopped[p]:
                continue
            sch = scheds[p]
            for ls in range(m):
                s = p * m + ls
                while slot_sample[s] < 0:
                    i = sch.next(ls)
                    if i < 0:
                        break
                    if reuse and Ls[p][i] <= reuse:  # finished within its probe tokens
                        sch.done(ls)
                        continue
                    ctx.refill_slot(s, p, i)
                    slot_sample[s] = i
                    slot_len[s] = reuse

    fill()
    step = 0
    while any(x >= 0 for x in slot_sample):
        if log is not None:
            log.append(tuple((s // m, slot_sample[s], slot_len[s] + 1) if slot_sample[s] >= 0 else None
                             for s in range(S)))
        decode = entries[entry_of(step)]
        if decode is None:
            ctx.decode_step_layers(*provide(step, 0))
        else:
            for layer in range(num_layers):
                decode(layer, *provide(step, layer))
        ctx.end_step()
        if after_step is not None:
            after_step(step)
        step += 1
        for s in range(S):
            i = slot_sample[s]
            if i < 0:
                continue
            slot_len[s] += 1
            p = s // m
            if slot_len[s] == Ls[p][i]:
                ctx.retire_slot(s)
                scheds[p].done(s - p * m)
                slot_sample[s] = -1
                if not stopped[p]:
                    done[p].append(i)
                    stopped[p] = stop_after is not None and len(done[p]) >= stop_after
        for p in range(NP):
            if stopped[p]:
                for s in range(p * m, (p + 1) * m):
                    if slot_sample[s] >= 0:
                        ctx.retire_slot(s)
                        scheds[p].done(s - p * m)
                        slot_sample[s] = -1
        fill()
    if accepted is not None:
        accepted.extend(done)
    return step


def plan_steps(cfg, lengths, policy: str, pred=None, stop_after=None, accepted=None, reuse=0,
               probe_log=None) -> list:
    """Step log of a group decode, from a dry-run context (bookkeeping only, no GPU).
    reuse = k runs the probe phase of prefix reuse first (its log into probe_log)."""
    ctx = context_for(cfg, dry_run=True, probe_tokens=reuse)
    for p in range(cfg.num_prompts):
        for layer in range(cfg.layers):
            ctx.prefill_shared(p, layer, cfg.prompt_lens[p], None, None)
    log = []
    nothing = (None, None, None, None)
    if reuse:
        probe_group(ctx, lengths, reuse, cfg.layers, lambda *a: nothing, log=probe_log)
    decode_group(ctx, schedulers_for(cfg, policy, pred), lengths, cfg.layers, lambda s, l: nothing, log=log,
                 stop_after=stop_after, accepted=accepted, reuse=reuse)
    ctx.destroy()
    return log
