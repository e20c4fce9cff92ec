"""GPU: the prefix store and the response pages hold exactly the K/V rows they
were given (read back through the C ABI, compared bit for bit), for the plain
and the MFMA-swizzled prefix layouts and for pages written by the append."""

import numpy as np
import pytest

from tests.gpu_harness import check_against_oracle, run_gpu_group, say
from workload import Workload, get_config

pytestmark = pytest.mark.gpu

CASES = [
    ("tiny_f32", {}),                                                     # fp32, plain layout
    ("qwen3_1p7b_l1_g32", {}),                                            # bf16, MFMA layout (16 rows)
    ("qwen3_1p7b_l1_g32", {"slots_per_prompt": 1, "samples_per_prompt": 6}),  # bf16, plain layout (2 rows)
    ("qwen3_8b_4prompts", {"layers": 2, "prompt_lens": (0, 77, 300), "samples_per_prompt": 12,
                           "length_dist": ("lognormal", 3.5, 1.0, 1, 100), "max_suffix_len": 100,
                           "pool_rows": None}),                               # 64 rows, three prompts
]


def _bits(wl, kind, idx):
    a = wl.pool(kind)[np.asarray(idx, dtype=np.int64)]
    return a.view(np.uint16) if a.dtype == np.uint16 else a.view(np.uint32)


@pytest.mark.parametrize("name,over", CASES)
def test_stores_round_trip(name, over):
    cfg = get_config(name).with_(**over) if over else get_config(name)
    cfg = cfg.with_(samples_per_prompt=min(cfg.samples_per_prompt, 12))
    wl = Workload(cfg)
    checked = {"prefix": 0, "response": 0}

    def inspect(ctx, step, log):
        if step == 0:
            for p in range(cfg.num_prompts):
                for layer in range(cfg.layers):
                    k, v = ctx.read_prefix(p, layer, cfg.prompt_lens[p])
                    idx = wl.prefix_index(layer, p)
                    assert np.array_equal(k.view(_bits(wl, "k", idx).dtype), _bits(wl, "k", idx)), (p, layer)
                    assert np.array_equal(v.view(_bits(wl, "v", idx).dtype), _bits(wl, "v", idx)), (p, layer)
                    checked["prefix"] += 1
        if step % 23 != 3:
            return
        for s, e in enumerate(log[step]):
            if e is None or s % 3:
                continue
            p, i, t = e
            if t == wl.L[p, i]:
                continue  # finished this step: already retired
            for layer in range(cfg.layers):
                k, v = ctx.read_response(s, layer)
                assert k.shape[0] == t
                idx = wl.suffix_index(layer, p, i, np.arange(t))
                assert np.array_equal(k.view(_bits(wl, "k", idx).dtype), _bits(wl, "k", idx)), (s, layer, t)
                assert np.array_equal(v.view(_bits(wl, "v", idx).dtype), _bits(wl, "v", idx)), (s, layer, t)
                checked["response"] += 1

    run_gpu_group(cfg, "fifo", capture=lambda k: False, wl=wl, inspect=inspect)
    say(f"  [{name}] {checked['prefix']} prefix and {checked['response']} response read-backs bit-exact")
    assert checked["prefix"] > 0 and checked["response"] > 0


def test_fp8_quantization_of_every_bf16_value():
    # The FP8 cache stores round-to-nearest-even E4M3 codes, saturating at
    # +-448: prefill K and V with every finite bf16 bit pattern and compare the
    # stored codes with the oracle's rounding, code by code.
    import torch
    from oracle import encode_e4m3, round_e4m3
    from paper_2506_22950_amd.group import context_for
    from workload import bf16_bits_to_f64

    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    finite = ((bits >> 7) & 0xFF) != 0xFF
    bits = bits[finite]
    cfg = get_config("qwen3_1p7b_l1_g32").with_(prompt_lens=(64,), max_suffix_len=16)
    row = cfg.num_kv_heads * cfg.head_dim
    n = -(-len(bits) // row) * row
    k = np.resize(bits, n)
    v = np.resize(bits[::-1], n)
    P = n // row
    cfg = cfg.with_(prompt_lens=(P,))
    ctx = context_for(cfg, stream=torch.cuda.current_stream(), kv_fp8=True)
    kd = torch.from_numpy(k.view(np.int16).reshape(P, cfg.num_kv_heads, cfg.head_dim)).cuda()
    vd = torch.from_numpy(v.view(np.int16).reshape(P, cfg.num_kv_heads, cfg.head_dim)).cuda()
    ctx.prefill_shared(0, 0, P, kd, vd)
    gk, gv = ctx.read_prefix(0, 0, P)
    table = {}
    for name, src, got in (("K", k, gk), ("V", v, gv)):
        vals = bf16_bits_to_f64(src)
        want = np.array([encode_e4m3(x) for x in round_e4m3(vals)], dtype=np.uint8)
        bad = np.flatnonzero(got.reshape(-1) != want)
        assert len(bad) == 0, (name, [(hex(int(src[i])), hex(int(got.reshape(-1)[i])), hex(int(want[i])))
                                      for i in bad[:8]])
        table[name] = len(src)
    say(f"  E4M3 codes of {table['K']} + {table['V']} bf16 values bit-exact")
    ctx.destroy()


def test_fp8_append_codes():
    # Pages written by the append hold the E4M3 codes of the new rows.
    from oracle import encode_e4m3, round_e4m3
    from workload import bf16_bits_to_f64
    cfg = get_config("qwen3_1p7b_l1_g32").with_(samples_per_prompt=10, length_dist=("uniform", 1, 60),
                                                max_suffix_len=60)
    wl = Workload(cfg)
    seen = [0]

    def codes(kind, idx):
        vals = bf16_bits_to_f64(wl.pool(kind)[np.asarray(idx, dtype=np.int64)])
        return np.vectorize(encode_e4m3, otypes=[np.uint8])(round_e4m3(vals))

    def inspect(ctx, step, log):
        if step % 5 != 2:
            return
        for s, e in enumerate(log[step]):
            if e is None or e[2] == wl.L[e[0], e[1]]:
                continue
            p, i, t = e
            k, v = ctx.read_response(s, 0)
            idx = wl.suffix_index(0, p, i, np.arange(t))
            assert np.array_equal(k, codes("k", idx)) and np.array_equal(v, codes("v", idx)), (s, t)
            seen[0] += 1

    run_gpu_group(cfg, "fifo", capture=lambda j: False, wl=wl, inspect=inspect, kv_fp8=True)
    assert seen[0] > 0


def test_merge_timeout_is_reported():
    # The merge's bounded wait: with the bound forced to "give up at once"
    # from the host, every merge work-group writes NaN and returns (the
    # producers still finish), the next synchronising call reports E_DEVICE
    # and the context refuses further work.
    import torch
    from paper_2506_22950_amd import infs
    from paper_2506_22950_amd.group import context_for
    from workload.staging import DeviceInputs
    cfg = get_config("tiny_f32")
    wl = Workload(cfg)
    dev = DeviceInputs(wl)
    ctx = context_for(cfg, stream=torch.cuda.current_stream())
    k, v = dev.prefix(0, 0)
    ctx.prefill_shared(0, 0, cfg.prompt_lens[0], k, v)
    ctx.refill_slot(0, 0, 0)
    S = cfg.num_slots
    q = torch.zeros((S, cfg.num_q_heads, cfg.head_dim), dtype=torch.float32, device="cuda")
    kn = torch.zeros((S, cfg.num_kv_heads, cfg.head_dim), dtype=torch.float32, device="cuda")
    o = torch.zeros((S, cfg.num_q_heads, cfg.head_dim), dtype=torch.float32, device="cuda")
    ctx.set_merge_wait(-1)
    ctx.decode_step(0, q, kn, kn, o)
    ctx.end_step()
    with pytest.raises(infs.InfsError) as ei:
        ctx.sync()
    assert ei.value.status == infs.E_DEVICE
    assert torch.isnan(o[0]).all() and not o[1:].any()
    for _ in range(3):  # every later call names the original cause, once
        with pytest.raises(infs.InfsError) as ei:
            ctx.retire_slot(0)
        assert ei.value.status == infs.E_DEVICE
        msg = str(ei.value)
        assert msg.count("gave up waiting") == 1 and msg.count("unusable") == 1, msg
    ctx.destroy()


@pytest.mark.parametrize("case", ["bf16", "reuse", "fp8"])
def test_exchange_modes_agree_bitwise(case):
    # The XCD-local exchange of partials (the default for 8 KV heads on this
    # device) and the exchange through the coherence point move the same
    # values: every output agrees bit for bit (decode, probe launches, E4M3
    # cache), and the outputs match the oracle.
    cfg = get_config("qwen3_1p7b_g64").with_(layers=2, prompt_lens=(700,), samples_per_prompt=24,
                                             length_dist=("lognormal", 4.0, 1.0, 1, 300), max_suffix_len=300,
                                             pool_rows=None)
    reuse = 8 if case == "reuse" else 0
    kv8 = case == "fp8"
    wl = Workload(cfg)
    modes = {}

    def seen(ctx, step, log):
        modes.setdefault("default", ctx.exchange_mode())

    runs = []
    for exchange in (None, 0):
        probe = {} if reuse else None
        _, log, _, cap, _, _ = run_gpu_group(cfg, "sjf", wl=wl, split=128, inspect=seen, exchange=exchange,
                                             reuse=reuse, probe=probe, kv_fp8=kv8)
        runs.append((log, cap, probe))
    assert modes["default"] == 1, "8 KV heads on this device should exchange partials through the XCD's L2"
    (log1, cap1, pr1), (log0, cap0, pr0) = runs
    assert log1 == log0 and cap1.keys() == cap0.keys()
    for k in cap0:
        assert np.array_equal(cap1[k], cap0[k]), k
    if reuse:
        for j in pr0["captured"]:
            assert np.array_equal(pr1["captured"][j], pr0["captured"][j]), j
    check_against_oracle(cfg, wl, log0, {k: cap0[k] for k in list(cap0)[::5]}, kv_fp8=kv8)


def test_exchange_mode_guard():
    # Two KV heads span several XCDs: no XCD-local exchange.  With 8 heads,
    # mode 2 makes every work-group's XCD check fail: the next synchronising
    # call reports E_DEVICE and the context refuses further work.
    import torch
    from paper_2506_22950_amd import infs
    from paper_2506_22950_amd.group import context_for
    from workload.staging import DeviceInputs
    ctx = context_for(get_config("tiny_f32"), stream=torch.cuda.current_stream())
    assert ctx.exchange_mode() == 0
    with pytest.raises(infs.InfsError) as ei:
        ctx.set_exchange(1)
    assert ei.value.status == infs.E_STATE
    ctx.destroy()

    cfg = get_config("qwen3_1p7b_l1_g32")
    wl = Workload(cfg)
    dev = DeviceInputs(wl)
    ctx = context_for(cfg, stream=torch.cuda.current_stream())
    k, v = dev.prefix(0, 0)
    ctx.prefill_shared(0, 0, cfg.prompt_lens[0], k, v)
    ctx.refill_slot(0, 0, 0)
    S = cfg.num_slots
    q = torch.zeros((S, cfg.num_q_heads, cfg.head_dim), dtype=torch.bfloat16, device="cuda")
    kn = torch.zeros((S, cfg.num_kv_heads, cfg.head_dim), dtype=torch.bfloat16, device="cuda")
    o = torch.zeros((S, cfg.num_q_heads, cfg.head_dim), dtype=torch.float32, device="cuda")
    ctx.set_exchange(2)
    assert ctx.exchange_mode() == 2
    ctx.decode_step(0, q, kn, kn, o)
    ctx.end_step()
    with pytest.raises(infs.InfsError) as ei:
        ctx.sync()
    assert ei.value.status == infs.E_DEVICE and "another XCD" in str(ei.value)
    with pytest.raises(infs.InfsError) as ei:
        ctx.retire_slot(0)
    assert ei.value.status == infs.E_DEVICE
    ctx.destroy()
