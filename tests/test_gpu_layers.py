"""GPU parity of the step launch through every layer (infs_decode_step_layers).

Each case decodes a whole group with one launch per running step and checks,
against the float64 oracle: the step log and the device token counters bit
for bit, every captured output within the tolerance (1e-2 bf16, 1e-5 fp32),
idle rows exactly 0.  The default work split cuts responses into near-equal
pieces; each case is decoded again with the per-layer launch's chunks
(infs_set_step_split(ctx, 0)), checked against the oracle too, and with one
launch per layer (infs_decode_step): those two differ only in the order in
which a merge folds the split-K partials, so their outputs agree to float
rounding.
"""

import numpy as np
import pytest

from paper_2506_22950_amd import infs
from tests.gpu_harness import check_against_oracle, oracle_log, run_gpu_group, sample_steps, say
from workload import Workload, get_config

pytestmark = pytest.mark.gpu


def _layers_case(cfg, policy, split=128, every=2, layers=None, kv_fp8=False, window=1024, against_layer_path=True,
                 entry="decode_step_layers", scale=0.0):
    wl = Workload(cfg)
    want = oracle_log(cfg, wl, policy)
    cap = sample_steps(want, every=every, edge=2, refills=8).__contains__
    _, log, steps, captured, tokens, stats = run_gpu_group(cfg, policy, wl=wl, split=split, capture=cap,
                                                           kv_fp8=kv_fp8, window=window, entry=entry, scale=scale)
    assert log == want and steps == len(want), "step log differs from the oracle simulator"
    assert np.array_equal(tokens, wl.L), "device token counters differ from the drawn lengths"
    if entry == "decode_step_layers":
        assert stats.launches == steps, "one launch per running step"
    worst, n = check_against_oracle(cfg, wl, want, captured, layers=layers, kv_fp8=kv_fp8,
                                    scale=scale if scale > 0 else None)
    diff = 0.0
    if against_layer_path:
        _, log0, _, chunked, _, _ = run_gpu_group(cfg, policy, wl=wl, split=split, capture=cap, kv_fp8=kv_fp8,
                                                  window=window, entry=entry, scale=scale, step_split=0)
        assert log0 == want
        worst0, _ = check_against_oracle(cfg, wl, want, chunked, layers=layers, kv_fp8=kv_fp8,
                                         scale=scale if scale > 0 else None)
        worst = max(worst, worst0)
        _, _, _, per_layer, _, _ = run_gpu_group(cfg, policy, wl=wl, split=split, capture=cap, kv_fp8=kv_fp8,
                                                 window=window, scale=scale)
        for k in chunked:
            diff = max(diff, float(np.abs(chunked[k].astype(np.float64) - per_layer[k]).max()))
        assert diff <= 1e-5, f"step launch (per-layer chunks) and per-layer launches differ by {diff:.3g}"
    say(f"  [{cfg.name} {policy} step launch] {steps} steps, {n} outputs vs oracle max err {worst:.3g} "
        f"(both work splits); per-layer chunks vs per-layer launches {diff:.3g}")


_BF16_SMALL = dict(prompt_lens=(700,), samples_per_prompt=24, length_dist=("lognormal", 4.0, 1.0, 1, 300),
                   max_suffix_len=300, pool_rows=None)


def test_step_launch_bf16_mfma32_four_layers():
    # The throughput workload's shape (16Q/8KV, d=128, m=16: 32 prefix rows on MFMA
    # tiles) with four layers, so that layers wait on their predecessors.
    _layers_case(get_config("qwen3_1p7b_g64").with_(layers=4, **_BF16_SMALL), "sjf")


def test_step_launch_f32_wave_every_step():
    # fp32 wavefront path, three layers, three prefix chunks, responses to 400.
    cfg = get_config("tiny_f32").with_(layers=3, prompt_lens=(300,), length_dist=("uniform", 1, 400),
                                       max_suffix_len=400)
    _layers_case(cfg, "fifo", every=1)


def test_step_launch_hpk4_three_prompts():
    # 32Q/8KV (64 prefix rows per prompt), three prompts including an empty prefix:
    # each prompt's layers wait only on that prompt's merges.
    cfg = get_config("qwen3_8b_4prompts").with_(layers=3, prompt_lens=(0, 130, 511), samples_per_prompt=20,
                                                length_dist=("lognormal", 4.0, 1.0, 1, 260), max_suffix_len=260,
                                                pool_rows=None)
    _layers_case(cfg, "sjf", every=3)


def test_step_launch_bf16_wave_single_slot():
    # m=1: 2 prefix rows on the bf16 wavefront path.
    cfg = get_config("qwen3_1p7b_l1_g32").with_(layers=3, slots_per_prompt=1, samples_per_prompt=4,
                                                prompt_lens=(257,), length_dist=("lognormal", 4.0, 0.8, 1, 300),
                                                max_suffix_len=300)
    _layers_case(cfg, "fifo", every=5)


def test_step_launch_wide_scores_and_scale():
    # Wide score ranges (see test_gpu_parity) and a non-default scale through the step launch.
    cfg = get_config("qwen3_1p7b_g64").with_(layers=3, **_BF16_SMALL, qk_scale=(8.0, 0.1, 8.0))
    _layers_case(cfg, "sjf", every=3)
    _layers_case(get_config("qwen3_1p7b_g64").with_(layers=2, **_BF16_SMALL), "sjf", every=3, scale=1.0)


def test_step_launch_fp8_cache():
    cfg = get_config("qwen3_1p7b_g64").with_(layers=3, **_BF16_SMALL)
    _layers_case(cfg, "sjf", every=3, kv_fp8=True)


def test_step_launch_alternating_with_layer_launches():
    # Step launches and per-layer launches mixed step by step in one context:
    # the arrival counters and page tables they share stay consistent.
    cfg = get_config("qwen3_1p7b_g64").with_(layers=3, **_BF16_SMALL)
    _layers_case(cfg, "sjf", every=2, entry=lambda step: "decode_step_layers" if step % 2 else "decode_step")


@pytest.mark.parametrize("name,every,window,kv_fp8", [
    ("qwen3_1p7b_g64", 397, 512, False),
    ("qwen3_1p7b_g64", 397, 512, True),
    ("longtail_g128", 997, 256, False),
    ("qwen3_8b_4prompts", 1201, 128, False),
], ids=["qwen3_1p7b_g64", "qwen3_1p7b_g64_e4m3", "longtail_g128", "qwen3_8b_4prompts"])
def test_step_launch_full_size_sampled(name, every, window, kv_fp8):
    # Whole workload, one step launch per running step (the benchmark's
    # configuration, with the bf16 cache and, for the benchmark workload, the
    # E4M3 cache); sampled steps on the first, middle and last layer.
    cfg = get_config(name)
    _layers_case(cfg, cfg.policy, split=0, every=every, layers=(0, cfg.layers // 2, cfg.layers - 1),
                 window=window, against_layer_path=False, kv_fp8=kv_fp8)


def test_step_launch_wait_give_up_is_reported():
    # Every wait of the step launch bounded: forced to give up at once from the
    # host, merges write NaN, the launch runs to its end, and the next
    # synchronising call reports E_DEVICE.
    import torch

    from paper_2506_22950_amd.group import context_for
    from workload.staging import DeviceInputs

    cfg = get_config("qwen3_1p7b_g64").with_(layers=3, **_BF16_SMALL)
    wl = Workload(cfg)
    dev = DeviceInputs(wl)
    ctx = context_for(cfg, stream=torch.cuda.current_stream())
    assert ctx.step_launch_workgroups > 0
    keep = []
    for layer in range(cfg.layers):
        k, v = dev.prefix(layer, 0)
        keep.append((k, v))
        ctx.prefill_shared(0, layer, cfg.prompt_lens[0], k, v)
    ctx.refill_slot(0, 0, 0)
    ctx.refill_slot(3, 0, 1)
    L, S, Hq, Hkv, d = cfg.layers, cfg.num_slots, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim
    q = torch.zeros((L, S, Hq, d), dtype=torch.int16, device="cuda")
    kn = torch.zeros((L, S, Hkv, d), dtype=torch.int16, device="cuda")
    o = torch.zeros((L, S, Hq, d), dtype=torch.float32, device="cuda")
    ctx.set_merge_wait(-1)
    ctx.decode_step_layers(q, kn, kn, o)
    ctx.end_step()
    with pytest.raises(infs.InfsError) as ei:
        ctx.sync()
    assert ei.value.status == infs.E_DEVICE
    assert torch.isnan(o[:, 0]).all() and torch.isnan(o[:, 3]).all()
    assert not o[:, 1].any() and not o[:, 2].any()
    ctx.destroy()


@pytest.mark.parametrize("kv_fp8", [False, True], ids=["bf16", "fp8"])
def test_step_launch_exchange_modes_agree_bitwise(kv_fp8):
    # The step launch exchanges split-K partials through the XCD's L2 when every
    # work-group of a KV head runs on one XCD (the default for 8 KV heads on
    # this device), else through the coherence point; both move the same
    # values, so every output agrees bit for bit, and matches the oracle.
    cfg = get_config("qwen3_1p7b_g64").with_(layers=3, **_BF16_SMALL)
    wl = Workload(cfg)
    modes = {}

    def seen(ctx, step, log):
        modes.setdefault("default", ctx.exchange_mode())

    runs = []
    for exchange in (None, 0):
        _, log, _, cap, _, _ = run_gpu_group(cfg, "sjf", wl=wl, split=128, inspect=seen, exchange=exchange,
                                             kv_fp8=kv_fp8, entry="decode_step_layers")
        runs.append((log, cap))
    assert modes["default"] == 1, "8 KV heads on this device should exchange partials through the XCD's L2"
    (log1, cap1), (log0, cap0) = runs
    assert log1 == log0 and cap1.keys() == cap0.keys()
    for k in cap0:
        assert np.array_equal(cap1[k], cap0[k]), k
    worst, n = check_against_oracle(cfg, wl, log0, {k: cap0[k] for k in list(cap0)[::5]}, kv_fp8=kv_fp8)
    say(f"  [step launch exchange modes {'fp8' if kv_fp8 else 'bf16'}] {len(cap0)} steps bitwise equal; "
        f"{n} outputs vs oracle max err {worst:.3g}")


def test_step_launch_exchange_placement_check():
    # In the XCD-local exchange every work-group of the step launch checks that
    # it runs on the XCD the plan assumes; mode 2 makes that check fail on every
    # work-group: the launch runs to its end and the next synchronising call
    # reports E_DEVICE.
    import torch

    from paper_2506_22950_amd.group import context_for
    from workload.staging import DeviceInputs

    cfg = get_config("qwen3_1p7b_g64").with_(layers=2, **_BF16_SMALL)
    wl = Workload(cfg)
    dev = DeviceInputs(wl)
    ctx = context_for(cfg, stream=torch.cuda.current_stream())
    keep = []
    for layer in range(cfg.layers):
        k, v = dev.prefix(layer, 0)
        keep.append((k, v))
        ctx.prefill_shared(0, layer, cfg.prompt_lens[0], k, v)
    ctx.refill_slot(0, 0, 0)
    L, S, Hq, Hkv, d = cfg.layers, cfg.num_slots, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim
    q = torch.zeros((L, S, Hq, d), dtype=torch.int16, device="cuda")
    kn = torch.zeros((L, S, Hkv, d), dtype=torch.int16, device="cuda")
    o = torch.zeros((L, S, Hq, d), dtype=torch.float32, device="cuda")
    ctx.set_exchange(2)
    ctx.decode_step_layers(q, kn, kn, o)
    ctx.end_step()
    with pytest.raises(infs.InfsError) as ei:
        ctx.sync()
    assert ei.value.status == infs.E_DEVICE
    ctx.destroy()


def _probe_case(cfg, policy, k, split=128):
    # The probe phase with one launch per probe step (infs_probe_step_layers) against the
    # oracle, and against one launch per layer: with the per-layer chunks the two differ only
    # in the order the merges add partials.
    wl = Workload(cfg)
    want = oracle_log(cfg, wl, policy, reuse=k)
    runs = {}
    for entry, step_split in (("probe_step_layers", None), ("probe_step_layers", 0), ("probe_step", None)):
        probe = {}
        _, log, steps, _, tokens, stats = run_gpu_group(cfg, policy, wl=wl, split=split, reuse=k, probe=probe,
                                                        capture=lambda j: False, probe_entry=entry,
                                                        step_split=step_split)
        assert log == want and steps == len(want)
        assert np.array_equal(tokens, wl.L), "device token counters (probe + decode) differ from the lengths"
        runs[(entry, step_split)] = probe
    worst = 0.0
    for key in (("probe_step_layers", None), ("probe_step_layers", 0)):
        w, n = check_against_oracle(cfg, wl, runs[key]["log"], runs[key]["captured"])
        worst = max(worst, w)
    a, b = runs[("probe_step_layers", 0)]["captured"], runs[("probe_step", None)]["captured"]
    assert a.keys() == b.keys()
    diff = max(float(np.abs(a[j].astype(np.float64) - b[j]).max()) for j in a)
    assert diff <= 1e-5, f"probe step launch and per-layer probe launches differ by {diff:.3g}"
    say(f"  [{cfg.name} probe step launch k={k}] {len(runs[('probe_step', None)]['log'])} probe steps, "
        f"{n} outputs vs oracle max err {worst:.3g}; vs per-layer probe launches {diff:.3g}")


def test_probe_step_launch_bf16_128_row_tiles():
    # 40 samples x hpk 2 = 80 rows per KV head on 128-row MFMA tiles, three layers.
    cfg = get_config("qwen3_1p7b_g64").with_(layers=3, prompt_lens=(300,), samples_per_prompt=40,
                                             slots_per_prompt=8, length_dist=("lognormal", 3.5, 1.0, 1, 200),
                                             max_suffix_len=200, pool_rows=None)
    _probe_case(cfg, "sjf", 16)


def test_probe_step_launch_hpk4_two_prompts():
    # 32Q/8KV: batches of 32 samples = 128 rows per KV head; two prompts, each probed in turn.
    cfg = get_config("qwen3_8b_4prompts").with_(layers=2, prompt_lens=(200, 450), samples_per_prompt=36,
                                                length_dist=("lognormal", 3.5, 1.0, 1, 160), max_suffix_len=160,
                                                pool_rows=None)
    _probe_case(cfg, "fptas_sjf", 8)


def test_probe_step_launch_f32_wave():
    # fp32 wavefront path: batches of 8 samples (16 rows), three layers.
    _probe_case(get_config("tiny_f32").with_(layers=3), "fifo", 5, split=0)


def _count_cut_steps(cfg, log, nj, split, mfma):
    # Steps whose work split cuts the responses into near-equal pieces (the library's own plan;
    # on MFMA tiles the prefix comes in 128-token chunks unless those would give some producer
    # two items, then in 256-token chunks).
    split = split or 256
    scmax = -(-cfg.max_suffix_len // split)
    cut = 0
    for row in log:
        lens = [e[2] if e is not None else 0 for e in row]
        live = {e[0] for e in row if e is not None}
        psplit = 128 if mfma else split
        npi = sum(-(-cfg.prompt_lens[p] // psplit) for p in live)
        if mfma:
            r0, _ = infs.step_split_plan(nj, lens, npi, psplit, split, scmax, mode=0)
            if r0["items"] > r0["n_suf"] or r0["n_pre"] < npi:
                psplit = 256
                npi = sum(-(-cfg.prompt_lens[p] // psplit) for p in live)
        roles, _ = infs.step_split_plan(nj, lens, npi, psplit, split, scmax)
        cut += roles["cut"]
    return cut


@pytest.mark.parametrize("name", ["bf16_mfma", "e4m3_mfma", "f32_wave"])
def test_step_launch_cut_pieces_multi_round(name):
    # Long responses on few slots: the per-layer chunks outnumber the response work-groups, so
    # the step launch cuts the responses into pieces of several load rounds per wavefront
    # (MFMA tiles on bf16 and E4M3 pages, and the fp32 wavefront path); checked against the
    # oracle, and the test asserts that the cut path ran.
    kv_fp8 = name == "e4m3_mfma"
    if name in ("bf16_mfma", "e4m3_mfma"):
        cfg = get_config("qwen3_1p7b_g64").with_(layers=2, prompt_lens=(256,), samples_per_prompt=16,
                                                 slots_per_prompt=16, length_dist=("uniform", 900, 1400),
                                                 max_suffix_len=1400, pool_rows=None)
        split, every = 0, 37
    else:
        cfg = get_config("tiny_f32").with_(layers=2, num_q_heads=16, num_kv_heads=8, samples_per_prompt=12,
                                           slots_per_prompt=8, length_dist=("uniform", 1500, 2000),
                                           max_suffix_len=2000)
        split, every = 128, 61
    seen = {}

    def grab(ctx, step, log):
        if not seen:
            seen["nj"] = ctx.step_launch_workgroups // cfg.num_kv_heads
            seen["mfma"] = ctx.kernel_info()["mfma"]
            seen["log"] = log

    wl = Workload(cfg)
    want = oracle_log(cfg, wl, cfg.policy)
    cap = sample_steps(want, every=every, edge=2, refills=4).__contains__
    _, log, steps, captured, tokens, _ = run_gpu_group(cfg, cfg.policy, wl=wl, split=split, capture=cap,
                                                       entry="decode_step_layers", inspect=grab, kv_fp8=kv_fp8)
    assert log == want and np.array_equal(tokens, wl.L)
    ncut = _count_cut_steps(cfg, want, seen["nj"], split, seen["mfma"])
    assert ncut > 0, "no step took the cut path"
    worst, n = check_against_oracle(cfg, wl, want, captured, kv_fp8=kv_fp8)
    say(f"  [{name} cut pieces] {steps} steps ({ncut} cut), {n} outputs vs oracle max err {worst:.3g}")


@pytest.mark.parametrize("rows,kv_fp8", [(16, False), (128, False), (16, True), (128, True)],
                         ids=["16_bf16", "128_bf16", "16_fp8", "128_fp8"])
def test_step_launch_prefix_tile_shapes(rows, kv_fp8):
    # The step launch's prefix chunks on the 16-row tile (four token groups; four prompts of
    # 700, 300, 500 and 400 tokens, responses of about 300 tokens, so that the chunks outnumber
    # the producers) and the 128-row tile (one token group walking the chunk; one prompt of 700
    # tokens), with partial last chunks, bf16 and E4M3 caches: 256-token chunks wherever the
    # 128-token ones would give some producer two items; against the oracle and, with the
    # per-layer partition, against per-layer launches.  The test asserts that some step took the
    # longer chunks.
    m = rows // 2  # hpk = 2
    if rows == 16:
        prompts, dist, longest, every = (700, 300, 500, 400), ("lognormal", 5.7, 0.2, 1, 400), 400, 15
    else:
        prompts, dist, longest, every = (700,), ("lognormal", 3.5, 1.0, 1, 200), 200, 5
    cfg = get_config("qwen3_1p7b_g64").with_(layers=2, prompt_lens=prompts, samples_per_prompt=m + 4,
                                             slots_per_prompt=m, length_dist=dist, max_suffix_len=longest,
                                             pool_rows=None)
    seen = {}

    def grab(ctx, step, log):
        if not seen:
            seen["nj"] = ctx.step_launch_workgroups // cfg.num_kv_heads

    wl = Workload(cfg)
    want = oracle_log(cfg, wl, "sjf")
    run_gpu_group(cfg, "sjf", wl=wl, split=128, capture=lambda k: False, kv_fp8=kv_fp8, stop_after=1,
                  entry="decode_step_layers", inspect=grab)
    nj = seen["nj"]
    longer = 0
    for row in want:
        lens = [e[2] if e is not None else 0 for e in row]
        live = {e[0] for e in row if e is not None}
        npi = sum(-(-cfg.prompt_lens[p] // 128) for p in live)
        r0, _ = infs.step_split_plan(nj, lens, npi, 128, 128, -(-cfg.max_suffix_len // 128), mode=0)
        longer += r0["items"] > r0["n_suf"] or r0["n_pre"] < npi
    assert longer > 0, "no step took the longer prefix chunks"
    say(f"  [{rows}-row prefix tile] {longer} of {len(want)} steps take 256-token prefix chunks")
    _layers_case(cfg, "sjf", every=every, kv_fp8=kv_fp8)
