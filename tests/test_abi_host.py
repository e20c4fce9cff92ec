"""Host-side checks of the C ABI (no GPU needed).

* libinfs.so loads and exports every function include/infs.h declares;
* the refill scheduler plus the context's slot bookkeeping (dry-run contexts)
  reproduce the oracle simulator's step logs bit for bit;
* every argument and state error is reported synchronously with its code.
"""

import os
import re

import numpy as np
import pytest

from oracle import POLICIES, simulate, simulate_group
from paper_2506_22950_amd import infs
from paper_2506_22950_amd.group import context_for, decode_group, plan_steps, schedulers_for
from tests.shape_table import ENTRIES as SHAPE_ENTRIES
from tests.shape_table import case_for
from tests.shape_table import case_id as shape_case_id
from workload import CONFIGS, Workload, get_config

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "infs.h")


def test_exports_every_declared_symbol():
    lib = infs.load()
    declared = set(re.findall(r"^\s*(?:[\w\s\*]+?)\b(infs_\w+)\s*\(", open(HEADER).read(), re.M))
    assert declared == set(infs.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name
    assert lib.infs_abi_version() == 3


def _oracle_log(cfg, L, policy, pred):
    """Oracle step log in the format of group.plan_steps: per step, per slot (p, i, t) or None."""
    total, res = simulate_group(L, cfg.slots_per_prompt, policy, pred)
    m = cfg.slots_per_prompt
    log = []
    for k in range(total):
        row = []
        for p, r in enumerate(res):
            for ls in range(m):
                e = r.log[k][ls] if k < r.steps else None
                row.append(None if e is None else (p, e[0], e[1]))
        log.append(tuple(row))
    return log


@pytest.mark.parametrize("policy", POLICIES)
def test_dry_run_step_log_matches_simulator_worked_example(policy):
    import json
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "sim_worked_example.json")))
    cfg = get_config("tiny_f32").with_(samples_per_prompt=g["G"], slots_per_prompt=g["m"], max_suffix_len=16)
    L = np.array([g["L"]])
    pred = np.array([g["pred"]], dtype=float)
    log = plan_steps(cfg, L, policy, pred)
    assert len(log) == g["policies"][policy]["steps"]
    assert log == _oracle_log(cfg, L, policy, pred)


@pytest.mark.parametrize("policy", POLICIES)
def test_dry_run_step_log_matches_simulator_random(policy):
    rng = np.random.default_rng(7)
    for trial in range(60):
        NP = int(rng.integers(1, 4))
        m = int(rng.integers(1, 6))
        G = int(rng.integers(1, 14))
        cfg = get_config("tiny_f32").with_(prompt_lens=tuple(int(x) for x in rng.integers(0, 40, NP)),
                                           samples_per_prompt=G, slots_per_prompt=m, max_suffix_len=40)
        L = rng.integers(1, 41, size=(NP, G))
        pred = L * np.exp(rng.normal(0, 0.3, size=L.shape))
        assert plan_steps(cfg, L, policy, pred) == _oracle_log(cfg, L, policy, pred), (trial, NP, m, G)


@pytest.mark.parametrize("name", list(CONFIGS))
def test_dry_run_full_workloads(name):
    # Full-size bookkeeping of every preset: step counts and logs equal the
    # simulator's, every sample decodes exactly its length, and continuous
    # refill needs fewer steps than naive micro groups.
    cfg = get_config(name)
    wl = Workload(cfg)
    log = plan_steps(cfg, wl.L, cfg.policy, wl.L_hat)
    assert log == _oracle_log(cfg, wl.L, cfg.policy, wl.L_hat)
    naive = plan_steps(cfg, wl.L, "naive", wl.L_hat)
    assert len(log) < len(naive)
    tokens = np.zeros_like(wl.L)
    for row in log:
        for e in row:
            if e is not None:
                tokens[e[0], e[1]] += 1
    assert np.array_equal(tokens, wl.L)


def _dry(**over):
    cfg = get_config("tiny_f32").with_(**over) if over else get_config("tiny_f32")
    ctx = context_for(cfg, dry_run=True)
    return cfg, ctx


def _code(fn, *a):
    with pytest.raises(infs.InfsError) as ei:
        fn(*a)
    return ei.value.status


def test_state_errors():
    cfg, ctx = _dry()
    none4 = (None, None, None, None)
    # decode of a live slot before its prompt is prefilled
    ctx.refill_slot(0, 0, 3)
    assert _code(ctx.decode_step, 0, *none4) == infs.E_STATE
    ctx.prefill_shared(0, 0, 32, None, None)
    assert _code(ctx.refill_slot, 0, 0, 4) == infs.E_STATE          # slot is live
    assert _code(ctx.refill_slot, 1, 0, 3) == infs.E_DUP            # id already dispatched
    assert _code(ctx.retire_slot, 1) == infs.E_STATE                # slot is empty
    assert _code(ctx.end_step) == infs.E_STATE                      # no layer decoded
    ctx.decode_step(0, *none4)
    assert _code(ctx.decode_step, 0, *none4) == infs.E_STATE        # same layer twice in a step
    assert _code(ctx.refill_slot, 1, 0, 5) == infs.E_STATE          # step is open
    assert _code(ctx.retire_slot, 0) == infs.E_STATE
    assert _code(ctx.prefill_shared, 0, 0, 32, None, None) == infs.E_STATE
    ctx.end_step()
    assert ctx.slot_state(0) == (3, 1)
    assert ctx.slot_state(1) == (-1, 0)
    ctx.retire_slot(0)
    assert ctx.slot_state(0) == (-1, 0)
    st = ctx.get_stats()
    assert (st.steps, st.launches, st.tokens) == (1, 1, 1)


def test_argument_errors():
    cfg, ctx = _dry()
    assert _code(ctx.refill_slot, 4, 0, 0) == infs.E_ARG    # slot out of range (S = 4)
    assert _code(ctx.refill_slot, 0, 1, 0) == infs.E_ARG    # prompt 1 does not exist
    assert _code(ctx.refill_slot, 0, 0, 8) == infs.E_ARG    # sample id >= G
    assert _code(ctx.refill_slot, 0, 0, -1) == infs.E_ARG
    assert _code(ctx.prefill_shared, 0, 1, 8, None, None) == infs.E_ARG   # layer out of range
    assert _code(ctx.prefill_shared, 0, 0, 33, None, None) == infs.E_ARG  # longer than max_prompt_len
    ctx.prefill_shared(0, 0, 8, None, None)
    assert _code(ctx.decode_step, 1, None, None, None, None) == infs.E_ARG
    assert _code(ctx.slot_state, 9) == infs.E_ARG
    assert _code(ctx.sample_tokens, 0) == infs.E_STATE        # no device counters in dry run


def test_capacity_errors():
    # Response longer than max_suffix_len.
    cfg, ctx = _dry(max_suffix_len=3)
    ctx.prefill_shared(0, 0, 32, None, None)
    ctx.refill_slot(0, 0, 0)
    none4 = (None, None, None, None)
    for _ in range(3):
        ctx.decode_step(0, *none4)
        ctx.end_step()
    assert _code(ctx.decode_step, 0, *none4) == infs.E_CAPACITY
    # Page pool too small: two slots need two pages, the pool has one.
    cfg = get_config("tiny_f32")
    ctx = context_for(cfg, dry_run=True, num_pages=1)
    ctx.prefill_shared(0, 0, 32, None, None)
    ctx.refill_slot(0, 0, 0)
    ctx.refill_slot(1, 0, 1)
    assert _code(ctx.decode_step, 0, *none4) == infs.E_CAPACITY
    ctx.retire_slot(1)
    ctx.decode_step(0, *none4)   # the failed attempt changed nothing; one page suffices now
    ctx.end_step()


def test_pages_recycled():
    # A slot's pages return to the pool on retire: with a pool of exactly one
    # slot's worth, consecutive samples can reuse it indefinitely.
    cfg = get_config("tiny_f32").with_(max_suffix_len=40)
    ctx = context_for(cfg, dry_run=True, num_pages=3)
    ctx.prefill_shared(0, 0, 32, None, None)
    none4 = (None, None, None, None)
    for i in range(8):
        ctx.refill_slot(0, 0, i)
        for _ in range(40):
            ctx.decode_step(0, *none4)
            ctx.end_step()
        ctx.retire_slot(0)


def test_create_validation():
    base = dict(num_layers=1, num_q_heads=4, num_kv_heads=2, head_dim=64, num_prompts=1, slots_per_prompt=4,
                samples_per_prompt=8, max_prompt_len=32, max_suffix_len=64, page_tokens=0, num_pages=0,
                split_tokens=0, dtype=infs.F32, scale=0.0, flags=infs.FLAG_DRY_RUN)
    infs.Context(infs.make_config(**base)).destroy()
    bad = [dict(num_q_heads=3), dict(head_dim=96), dict(num_prompts=0), dict(num_prompts=17),
           dict(slots_per_prompt=65), dict(samples_per_prompt=0), dict(max_suffix_len=0), dict(page_tokens=32),
           dict(split_tokens=100), dict(dtype=7), dict(scale=-1.0), dict(flags=2), dict(num_layers=0),
           dict(slots_per_prompt=16),   # fp32 with 32 prefix rows: no kernel
           # page table of 2^20 probe sequences x 512 pages = 2 GiB
           dict(samples_per_prompt=1 << 20, probe_tokens=1, max_suffix_len=1 << 13),
           # split-K workspace: 4 slots x 16 chunks x 2^16 KV heads x 2 rows x 64 floats, plus the prefix: > 2 GiB
           dict(num_q_heads=1 << 17, num_kv_heads=1 << 16, max_suffix_len=4096)]
    for b in bad:
        with pytest.raises(infs.InfsError) as ei:
            infs.Context(infs.make_config(**{**base, **b}))
        assert ei.value.status == infs.E_ARG, b
        assert infs.load().infs_last_error(None).decode() != "no error"


def test_sched_errors():
    s = infs.Sched(4, 2, "fifo")
    assert s.next(0) == 0
    with pytest.raises(infs.InfsError):
        s.next(0)           # slot already holds a sample
    with pytest.raises(infs.InfsError):
        s.done(1)           # slot 1 is empty
    with pytest.raises(infs.InfsError):
        s.next(2)           # slot out of range
    with pytest.raises(infs.InfsError):
        infs.Sched(4, 2, "sjf")   # SJF needs predictions
    with pytest.raises(infs.InfsError):
        infs.Sched(4, 2, "sjf", pred_len=[1.0, float("nan"), 2.0, 3.0])
    assert s.pending == 3


def test_fptas_assign_matches_oracle():
    # infs_fptas_assign (C++) and the oracle's Algorithm 2 (Python) agree on
    # the hand-worked cases and bit for bit on random predicted lengths.
    import json
    from oracle import fptas_assign
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "sim_worked_example.json")))
    for case in g["fptas_cases"]:
        group, pos = infs.fptas_assign(case["pred"], case["N"], case["eps"])
        assert list(group) == case["group"] and list(pos) == case["pos"], case["note"]
    rng = np.random.default_rng(11)
    for _ in range(2000):
        G = int(rng.integers(1, 70))
        N = int(rng.integers(1, 17))
        eps = float(rng.choice([0.01, 0.1, 0.25, 1.0]))
        pred = np.exp(rng.normal(5.5, 1.2, size=G))
        if rng.random() < 0.3:
            pred = np.round(pred)  # integer predictions: many equal sizes
        group, pos = infs.fptas_assign(pred, N, eps)
        want_g, want_p = fptas_assign(pred, N, eps)
        assert list(group) == want_g and list(pos) == want_p


def test_fptas_assign_errors():
    for args in (([1.0, 2.0], 0, 0.1), ([1.0, 2.0], 2, 0.0), ([1.0, float("nan")], 2, 0.1),
                 ([1.0, -1.0], 2, 0.1), ([0.0, 0.0], 2, 0.1), ([], 2, 0.1)):
        with pytest.raises(infs.InfsError):
            infs.fptas_assign(*args)
    for policy in ("fptas", "fptas_sjf", "lpt"):
        with pytest.raises(infs.InfsError):
            infs.Sched(4, 2, policy)  # these policies need predicted lengths


@pytest.mark.parametrize("policy", ["fixed_row", "fptas", "sjf", "fptas_sjf", "lpt"])
def test_dry_run_scheduler_policies_full_workload(policy):
    # The policies of the scheduler comparison on the benchmark workload's
    # lengths: step logs equal the simulator's.
    cfg = get_config("qwen3_1p7b_g64")
    wl = Workload(cfg)
    assert plan_steps(cfg, wl.L, policy, wl.L_hat) == _oracle_log(cfg, wl.L, policy, wl.L_hat)


def test_dry_run_dynamic_slot_matches_simulator():
    # Dynamic-slot sampling through the library (FIFO over a stream, stop
    # after `target` completions per prompt, in-flight samples discarded):
    # step logs and accepted samples equal the simulator's.
    from oracle import simulate_dynamic
    rng = np.random.default_rng(12)
    for trial in range(40):
        NP = int(rng.integers(1, 4))
        m = int(rng.integers(1, 6))
        target = int(rng.integers(1, 12))
        n = 4 * target + 10
        cfg = get_config("tiny_f32").with_(prompt_lens=tuple(int(x) for x in rng.integers(0, 40, NP)),
                                           samples_per_prompt=n, slots_per_prompt=m, max_suffix_len=40)
        L = rng.integers(1, 41, size=(NP, n))
        acc = []
        log = plan_steps(cfg, L, "fifo", None, stop_after=target, accepted=acc)
        res = [simulate_dynamic(L[p], m, target) for p in range(NP)]
        want = []
        for k in range(max(r.steps for r in res)):
            row = []
            for p, r in enumerate(res):
                for ls in range(m):
                    e = r.log[k][ls] if k < r.steps else None
                    row.append(None if e is None else (p, e[0], e[1]))
            want.append(tuple(row))
        assert log == want, trial
        assert acc == [r.accepted for r in res], trial



def _oracle_reuse_log(cfg, L, policy, pred, k):
    total, res = simulate_group(L, cfg.slots_per_prompt, policy, pred, reuse=k)
    m = cfg.slots_per_prompt
    return [tuple(None if (k2 >= r.steps or r.log[k2][ls] is None) else (p, r.log[k2][ls][0], r.log[k2][ls][1])
                  for p, r in enumerate(res) for ls in range(m)) for k2 in range(total)]


@pytest.mark.parametrize("policy", POLICIES)
def test_dry_run_prefix_reuse_matches_simulator(policy):
    # Probe phase of k tokens, then decode resuming at k+1: the library's step
    # log equals the simulator's with the same reuse; the probe log has, per
    # token position t <= k and batch, exactly the samples longer than t-1.
    rng = np.random.default_rng(15)
    for trial in range(30):
        NP = int(rng.integers(1, 3))
        m = int(rng.integers(1, 5))
        G = int(rng.integers(1, 20))
        k = int(rng.integers(1, 6))
        cfg = get_config("tiny_f32").with_(prompt_lens=tuple(int(x) for x in rng.integers(0, 40, NP)),
                                           samples_per_prompt=G, slots_per_prompt=m, max_suffix_len=30)
        L = rng.integers(1, 31, size=(NP, G))
        pred = L * np.exp(rng.normal(0, 0.3, size=L.shape))
        plog = []
        log = plan_steps(cfg, L, policy, pred, reuse=k, probe_log=plog)
        assert log == _oracle_reuse_log(cfg, L, policy, pred, k), (trial, NP, m, G, k)
        seen = {}
        for row in plog:
            for e in row:
                if e is not None:
                    p, i, t = e
                    assert t == seen.get((p, i), 0) + 1
                    seen[(p, i)] = t
        assert seen == {(p, i): min(int(L[p, i]), k) for p in range(NP) for i in range(G)}


def test_probe_state_machine_errors():
    cfg = get_config("tiny_f32").with_(samples_per_prompt=6, slots_per_prompt=2, max_suffix_len=16)
    ctx = context_for(cfg, dry_run=True, probe_tokens=2)
    assert ctx.probe_batch == 6
    ctx.prefill_shared(0, 0, cfg.prompt_lens[0], None, None)
    nothing = (None, None, None, None)
    assert _code(ctx.probe_step, 0, 0, 0, 7, None, *nothing) == infs.E_ARG         # batch too large
    assert _code(ctx.probe_step, 0, 0, 3, 4, None, *nothing) == infs.E_ARG         # past the last sample
    ctx.probe_step(0, 0, 0, 6, [1, 1, 1, 1, 0, 1], *nothing)
    assert _code(ctx.probe_step, 0, 0, 0, 6, [1] * 6, *nothing) == infs.E_STATE    # another batch in the step
    assert _code(ctx.decode_step, 0, *nothing) == infs.E_STATE                    # decode during a probe step
    assert _code(ctx.refill_slot, 0, 0, 0) == infs.E_STATE                        # refill during a probe step
    ctx.end_probe_step()
    assert [ctx.probe_state(0, i) for i in range(6)] == [1, 1, 1, 1, 0, 1]
    assert _code(ctx.end_probe_step) == infs.E_STATE                              # no step open
    ctx.probe_step(0, 0, 0, 6, None, *nothing)
    ctx.end_probe_step()
    assert _code(ctx.probe_step, 0, 0, 0, 1, None, *nothing) == infs.E_CAPACITY   # sample 0 has its k tokens
    ctx.refill_slot(0, 0, 0)
    assert ctx.slot_state(0) == (0, 2)                                            # resumes after the probe tokens
    assert _code(ctx.probe_step, 0, 0, 0, 1, None, *nothing) == infs.E_STATE      # already dispatched
    ctx.release_sample(0, 3)
    assert _code(ctx.release_sample, 0, 3) == infs.E_DUP
    assert _code(ctx.refill_slot, 1, 0, 3) == infs.E_DUP
    plain = context_for(cfg, dry_run=True)
    assert plain.probe_batch == 0
    assert _code(plain.probe_step, 0, 0, 0, 1, None, *nothing) == infs.E_STATE
    assert _code(plain.release_sample, 0, 0) == infs.E_STATE



def test_probe_step_launch_state_machine():
    # infs_probe_step_layers on a dry-run context: the whole probe step in one call, the same
    # bookkeeping as one infs_probe_step per layer, and its own argument and state errors.
    cfg = get_config("tiny_f32").with_(layers=3, samples_per_prompt=6, slots_per_prompt=2, max_suffix_len=16)
    nothing = (None, None, None, None)
    a = context_for(cfg, dry_run=True, probe_tokens=2)
    b = context_for(cfg, dry_run=True, probe_tokens=2)
    assert _code(a.probe_step_layers, 0, 0, 6, None, *nothing) == infs.E_STATE    # prompt not prefilled
    for ctx in (a, b):
        for layer in range(cfg.layers):
            ctx.prefill_shared(0, layer, cfg.prompt_lens[0], None, None)
    live = [1, 0, 1, 1, 1, 1]
    a.probe_step_layers(0, 0, 6, live, *nothing)
    for layer in range(cfg.layers):
        b.probe_step(layer, 0, 0, 6, live, *nothing)
    assert _code(a.probe_step_layers, 0, 0, 6, live, *nothing) == infs.E_STATE   # the step is probed
    assert _code(a.probe_step, 0, 0, 0, 6, live, *nothing) == infs.E_STATE
    a.end_probe_step()
    b.end_probe_step()
    assert [a.probe_state(0, i) for i in range(6)] == [b.probe_state(0, i) for i in range(6)] == live
    assert _code(a.probe_step_layers, 0, 0, 7, None, *nothing) == infs.E_ARG      # batch too large
    assert _code(a.probe_step_layers, 1, 0, 1, None, *nothing) == infs.E_ARG      # no prompt 1
    assert _code(a.probe_step_layers, 0, 0, 6, None, *nothing, 8, 0, 0) == infs.E_ARG  # stride below a layer
    a.probe_step(0, 0, 0, 6, None, *nothing)                                     # per-layer step open
    assert _code(a.probe_step_layers, 0, 0, 6, None, *nothing) == infs.E_STATE
    for layer in range(1, cfg.layers):
        a.probe_step(layer, 0, 0, 6, None, *nothing)
    a.end_probe_step()
    assert _code(a.probe_step_layers, 0, 0, 1, None, *nothing) == infs.E_CAPACITY  # sample 0 has its k tokens
    sa, sb = a.get_stats(), b.get_stats()
    assert (sa.launches, sb.launches) == (1 + cfg.layers, cfg.layers)  # a: one step launch, then per layer
    assert sa.tokens == sb.tokens + 6 and sa.alg_bytes > sb.alg_bytes
    plain = context_for(cfg, dry_run=True)
    assert _code(plain.probe_step_layers, 0, 0, 1, None, *nothing) == infs.E_STATE
    for ctx in (a, b, plain):
        ctx.destroy()


def test_fp8_kv_validation():
    # The FP8 cache needs bf16, head_dim 128 and the MFMA prefix path.
    for name, over in (("tiny_f32", {}),                                           # fp32
                       ("qwen3_1p7b_l1_g32", {"slots_per_prompt": 1}),            # 2 prefix rows
                       ("qwen3_1p7b_l1_g32", {"head_dim": 64})):                   # head_dim 64
        cfg = get_config(name).with_(**over)
        with pytest.raises(infs.InfsError) as ei:
            context_for(cfg, dry_run=True, kv_fp8=True)
        assert ei.value.status == infs.E_ARG
    ctx = context_for(get_config("qwen3_1p7b_g64"), dry_run=True, kv_fp8=True)
    ctx.destroy()


@pytest.mark.parametrize("entry", SHAPE_ENTRIES, ids=shape_case_id)
def test_kernel_selection_reaches_every_instantiation(entry):
    # Each instantiation is selected by its small workload (dry run, no GPU).
    cfg, probe, want = case_for(entry)
    ctx = context_for(cfg, dry_run=True, probe_tokens=probe, kv_fp8=entry[5])
    got = ctx.kernel_info()
    ctx.destroy()
    for k, v in want.items():
        assert got[k] == v, (k, got)


def test_exchange_mode_on_dry_run():
    # A dry-run context has no device, so no XCD-local exchange of partials.
    cfg, ctx = _dry()
    assert ctx.exchange_mode() == 0
    assert _code(ctx.set_exchange, 1) == infs.E_STATE
    assert _code(ctx.set_exchange, 2) == infs.E_STATE
    assert _code(ctx.set_exchange, 3) == infs.E_ARG
    ctx.set_exchange(0)
    assert ctx.exchange_mode() == 0
    ctx.destroy()


def test_step_split_mode_on_dry_run():
    # The step launch's work split: 0 or 1, not changed while a step is open.
    cfg, ctx = _dry()
    none4 = (None, None, None, None)
    assert _code(ctx.set_step_split, 2) == infs.E_ARG
    assert _code(ctx.set_step_split, -1) == infs.E_ARG
    ctx.set_step_split(0)
    ctx.set_step_split(1)
    ctx.prefill_shared(0, 0, 32, None, None)
    ctx.refill_slot(0, 0, 3)
    ctx.decode_step(0, *none4)
    assert _code(ctx.set_step_split, 0) == infs.E_STATE
    ctx.end_step()
    ctx.set_step_split(0)
    ctx.destroy()


def test_static_entry_point_workspace_limit():
    # infs_decode_step_static keeps the split-K workspace and counters in a
    # static array of INFS_STATIC_SCRATCH_BYTES: the benchmark and long-tail
    # groups fit; the four-prompt 8B-shaped group (about 68 MB of workspace) is
    # rejected with E_CAPACITY before anything changes, and the regular entry
    # point still decodes it.
    for name, fits in (("qwen3_1p7b_g64", True), ("longtail_g128", True), ("qwen3_8b_4prompts", False)):
        cfg = get_config(name)
        ctx = context_for(cfg, dry_run=True)
        for p in range(cfg.num_prompts):
            for layer in range(cfg.layers):
                ctx.prefill_shared(p, layer, cfg.prompt_lens[p], None, None)
        for s in range(cfg.num_slots):
            ctx.refill_slot(s, s // cfg.slots_per_prompt, s % cfg.slots_per_prompt)
        none4 = (None, None, None, None)
        if fits:
            ctx.decode_step_static(0, *none4)
        else:
            assert _code(ctx.decode_step_static, 0, *none4) == infs.E_CAPACITY
            assert "static scratch" in ctx.last_error
            assert ctx.get_stats().launches == 0
            ctx.decode_step(0, *none4)
        for layer in range(1, cfg.layers):
            ctx.decode_step(layer, *none4)
        ctx.end_step()
        assert ctx.get_stats().launches == cfg.layers


def test_sched_optimum_matches_oracle():
    # infs_sched_optimum (branch and bound) against the oracle's capacity
    # search on random small groups and on the scheduler study's groups the
    # oracle finishes; every schedule it returns must have its reported steps.
    from oracle import makespan, optimum
    from workload import SCHEDULER_STUDY, scheduler_study_lengths

    rng = np.random.default_rng(21)
    cases = []
    for _ in range(300):
        G = int(rng.integers(1, 13))
        cases.append((rng.integers(1, 60, size=G), int(rng.integers(1, 6))))
    for k, (_, mu, sigma) in enumerate(SCHEDULER_STUDY):
        L, _ = scheduler_study_lengths(mu, sigma, 8, 32, cap=1024, seed=k)
        cases.extend((row, 4) for row in L)
    checked = 0
    for L, m in cases:
        best, lower, slot = infs.sched_optimum(L, m)
        assert best == lower, (L, m)
        assert makespan(L, slot, m) == best
        want, _ = optimum(L, m, max_nodes=300_000)
        if want is not None:
            assert best == want, (L, m)
            checked += 1
    assert checked >= len(cases) - 4


def test_sched_optimum_budget_and_errors():
    best, lower, slot = infs.sched_optimum([7, 6, 5, 4, 3, 3, 2, 2, 1], 3, max_nodes=0)
    assert lower <= 11 <= best   # 33 / 3 = 11 is reached by 7+4 | 6+3+2 | 5+3+2+1
    assert infs.sched_optimum([7, 6, 5, 4, 3, 3, 2, 2, 1], 3)[:2] == (11, 11)
    for bad in (([0, 3], 2), ([3, 4], 0)):
        with pytest.raises(infs.InfsError):
            infs.sched_optimum(*bad)


def test_step_launch_state_machine():
    # infs_decode_step_layers on a dry-run context: one call decodes every
    # layer of a step (one launch, L layers of bytes), needs a step with no
    # layer decoded yet, checks its strides, and leaves the step for end_step.
    cfg = get_config("qwen3_1p7b_g64").with_(layers=3, prompt_lens=(200,), samples_per_prompt=8,
                                             length_dist=("uniform", 1, 40), max_suffix_len=40, pool_rows=None)
    ctx = context_for(cfg, dry_run=True)
    assert ctx.step_launch_workgroups == 0
    none4 = (None, None, None, None)
    ctx.refill_slot(0, 0, 0)
    for layer in range(2):
        ctx.prefill_shared(0, layer, 200, None, None)
    assert _code(ctx.decode_step_layers, *none4) == infs.E_STATE     # layer 2 not prefilled
    ctx.prefill_shared(0, 2, 200, None, None)
    assert _code(ctx.decode_step_layers, *none4, 16, 0, 0) == infs.E_ARG    # stride below one layer
    S, Hq, d = cfg.num_slots, cfg.num_q_heads, cfg.head_dim
    assert _code(ctx.decode_step_layers, *none4, S * Hq * d * 2 + 8, 0, 0) == infs.E_ARG  # not a multiple of 16
    ctx.decode_step_layers(*none4)
    assert _code(ctx.decode_step, 0, *none4) == infs.E_STATE         # every layer already decoded
    assert _code(ctx.decode_step_layers, *none4) == infs.E_STATE
    ctx.end_step()
    ctx.decode_step(0, *none4)
    assert _code(ctx.decode_step_layers, *none4) == infs.E_STATE     # a layer of this step is decoded
    ctx.decode_step(1, *none4)
    ctx.decode_step(2, *none4)
    ctx.end_step()
    st = ctx.get_stats()
    assert (st.steps, st.launches) == (2, 4)
    assert ctx.slot_state(0) == (0, 2)


def test_step_launch_dry_run_logs_match_layer_path():
    # Whole groups through decode_group with the step launch and with per-layer
    # launches: identical step logs and byte counts (the library counts the
    # same algorithmic bytes for both).
    cfg = get_config("qwen3_8b_4prompts").with_(layers=2, prompt_lens=(0, 130, 511), samples_per_prompt=12,
                                                length_dist=("lognormal", 3.5, 1.0, 1, 100), max_suffix_len=100,
                                                pool_rows=None)
    wl = Workload(cfg)
    out = {}
    for entry in ("decode_step", "decode_step_layers"):
        ctx = context_for(cfg, dry_run=True)
        for p in range(cfg.num_prompts):
            for layer in range(cfg.layers):
                ctx.prefill_shared(p, layer, cfg.prompt_lens[p], None, None)
        log = []
        decode_group(ctx, schedulers_for(cfg, "sjf", wl.L_hat), wl.L, cfg.layers, lambda s, l: (None,) * 4,
                     log=log, entry=entry)
        out[entry] = (log, ctx.get_stats())
    (la, sa), (lb, sb) = out["decode_step"], out["decode_step_layers"]
    assert la == lb
    assert sa.launches == cfg.layers * sb.launches == cfg.layers * len(la)
    assert sa.alg_bytes == sb.alg_bytes and sa.tokens == sb.tokens
