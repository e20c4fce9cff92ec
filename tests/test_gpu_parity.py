"""GPU parity: the HIP path through the C ABI against the float64 oracle.

Bookkeeping (step counts, step logs, device per-sample token counters) must be
bit-exact; attention outputs within 1e-5 (fp32) or 1e-2 (bf16 K/V, fp32
accumulation) max abs error; idle slots' rows exactly 0.
"""

import numpy as np
import pytest

from tests.gpu_harness import (check_against_oracle, oracle_dynamic_log, oracle_log, run_gpu_group, sample_steps,
                               say)
from workload import Workload, get_config

pytestmark = pytest.mark.gpu


def _run_and_check(cfg, policy, capture=None, layers=None, split=0, window=1024, kv_fp8=False, scale=0.0):
    wl = Workload(cfg)
    want_log = oracle_log(cfg, wl, policy)
    cap = capture(want_log).__contains__ if capture else (lambda k: True)
    wl, log, steps, captured, tokens, stats = run_gpu_group(cfg, policy, capture=cap, split=split,
                                                          window=window, wl=wl, kv_fp8=kv_fp8, scale=scale)
    assert log == want_log, "step log differs from the oracle simulator"
    assert steps == len(want_log)
    assert np.array_equal(tokens, wl.L), "device token counters differ from the drawn lengths"
    worst, n = check_against_oracle(cfg, wl, log, captured, layers=layers, kv_fp8=kv_fp8,
                                    scale=scale if scale > 0 else None)
    say(f"  [{cfg.name} {policy}] checked {n} (slot, layer) outputs over {len(captured)} steps, "
        f"max abs err {worst:.3g}")
    return wl, log, captured


@pytest.mark.parametrize("policy", ["naive", "fifo"])
def test_tiny_f32_every_step(policy):
    # 1 layer, 4Q/2KV, d=64, P=32, G=8, m=4, L~U[1,64], fp32: every output of every step.
    _run_and_check(get_config("tiny_f32"), policy)


def test_tiny_f32_multichunk_ragged():
    # fp32 wavefront path over several split-K chunks with ragged tails:
    # P=300 with 128-token chunks, responses up to 400.
    cfg = get_config("tiny_f32").with_(prompt_lens=(300,), length_dist=("uniform", 1, 400), max_suffix_len=400)
    _run_and_check(cfg, "fifo", split=128, capture=lambda log: sample_steps(log, every=3))


def test_qwen3_1layer_bf16_mfma16():
    # Qwen3-1.7B-shaped layer: 16Q/8KV, d=128, P=512, G=32, m=8 (16 prefix rows: MFMA), FIFO.
    cfg = get_config("qwen3_1p7b_l1_g32")
    _run_and_check(cfg, "fifo", capture=lambda log: sample_steps(log, every=11))


def test_bf16_mfma32_small_every_step():
    # The throughput workload's shape (16Q/8KV, d=128, m=16: 32 prefix rows) on a
    # small group: 2 layers, P=700 (ragged last MFMA block), 128-token chunks.
    cfg = get_config("qwen3_1p7b_g64").with_(layers=2, prompt_lens=(700,), samples_per_prompt=24,
                                             length_dist=("lognormal", 4.0, 1.0, 1, 300), max_suffix_len=300,
                                             pool_rows=None)
    _run_and_check(cfg, "sjf", split=128, capture=lambda log: sample_steps(log, every=2))


@pytest.mark.parametrize("split", [512, 4096])
def test_bf16_long_split_chunks(split):
    # Longer split-K response chunks (the limit is 4096 tokens): responses span
    # up to three chunks with ragged tails, prompt 1000 (ragged MFMA block).
    top = 2 * split + 300
    cfg = get_config("qwen3_1p7b_g64").with_(layers=1, prompt_lens=(1000,), samples_per_prompt=20,
                                             length_dist=("uniform", 1, top), max_suffix_len=top, pool_rows=None)
    _run_and_check(cfg, "sjf", split=split,
                   capture=lambda log: sample_steps(log, every=max(1, len(log) // 60), refills=20))


def test_f32_wave_split_1024():
    # fp32 wavefront path with 1024-token response chunks: responses up to 2500.
    cfg = get_config("tiny_f32").with_(prompt_lens=(200,), length_dist=("uniform", 1, 2500), max_suffix_len=2500)
    _run_and_check(cfg, "fifo", split=1024, capture=lambda log: sample_steps(log, every=40, refills=8))


def test_bf16_mfma64_and_hpk4_multi_prompt():
    # Qwen3-8B shape (32Q/8KV: 4 query heads per KV head, 64 prefix rows), three
    # prompts of different lengths including an empty prefix.
    cfg = get_config("qwen3_8b_4prompts").with_(layers=2, prompt_lens=(0, 130, 511), samples_per_prompt=20,
                                                length_dist=("lognormal", 4.0, 1.0, 1, 260),
                                                max_suffix_len=260, pool_rows=None)
    _run_and_check(cfg, "sjf", split=128, capture=lambda log: sample_steps(log, every=3))


@pytest.mark.parametrize("policy", ["fptas", "fptas_sjf"])
def test_bf16_fptas_schedules(policy):
    # The decode path under the FPTAS plans (Algorithm 2 alone, and followed
    # by shortest-job-first refill as in Algorithm 1): bookkeeping bit-exact
    # and outputs against the oracle.
    cfg = get_config("qwen3_1p7b_g64").with_(layers=2, prompt_lens=(300,), samples_per_prompt=20,
                                             length_dist=("lognormal", 4.0, 1.0, 1, 200), max_suffix_len=200,
                                             pool_rows=None)
    _run_and_check(cfg, policy, split=128, capture=lambda log: sample_steps(log, every=4))


def test_bf16_dynamic_slot_stream():
    # Dynamic-slot sampling (Section 3.2, mode 2): 8 slots draw from a stream
    # of 60 samples and stop after 16 completions, discarding the samples
    # still decoding.  Step log equal to the simulator's; device token
    # counters equal the tokens each sample decoded (discarded ones included).
    cfg = get_config("qwen3_1p7b_g64").with_(layers=2, prompt_lens=(250,), samples_per_prompt=60,
                                             slots_per_prompt=8, length_dist=("lognormal", 3.5, 1.0, 1, 150),
                                             max_suffix_len=150, pool_rows=None)
    wl = Workload(cfg)
    want = oracle_dynamic_log(cfg, wl, 16)
    _, log, steps, captured, tokens, _ = run_gpu_group(cfg, "fifo", wl=wl, split=128, stop_after=16,
                                                       capture=lambda k: k % 3 == 0 or k == len(want) - 1)
    assert log == want and steps == len(want)
    counts = np.zeros_like(wl.L)
    for row in log:
        for e in row:
            if e is not None:
                counts[e[0], e[1]] += 1
    assert np.array_equal(tokens, counts)
    worst, n = check_against_oracle(cfg, wl, log, captured)
    say(f"  [dynamic-slot] {steps} steps, checked {n} outputs, max abs err {worst:.3g}")


def _prefix_reuse(cfg, policy, k, split=128):
    wl = Workload(cfg)
    want = oracle_log(cfg, wl, policy, reuse=k)
    probe = {}
    _, log, steps, captured, tokens, _ = run_gpu_group(cfg, policy, wl=wl, split=split, reuse=k, probe=probe,
                                                       capture=lambda j: j % 3 == 0 or j == len(want) - 1)
    assert log == want and steps == len(want)
    assert np.array_equal(tokens, wl.L), "device token counters (probe + decode) differ from the lengths"
    worst_p, n_p = check_against_oracle(cfg, wl, probe["log"], probe["captured"])
    worst, n = check_against_oracle(cfg, wl, log, captured)
    say(f"  [{cfg.name} reuse k={k}] {len(probe['log'])} probe steps ({n_p} outputs, max err {worst_p:.3g}), "
        f"{steps} decode steps ({n} outputs, max err {worst:.3g})")


def test_bf16_prefix_reuse_probe_128_row_tiles():
    # Prefix reuse (Section 4): 40 samples decode 16 probe tokens together
    # (80 query rows per KV head: 128-row MFMA tiles, two per wavefront), then SJF
    # decode resumes each at token 17; samples shorter than 17 never take a slot.
    cfg = get_config("qwen3_1p7b_g64").with_(layers=2, prompt_lens=(300,), samples_per_prompt=40,
                                             slots_per_prompt=8, length_dist=("lognormal", 3.5, 1.0, 1, 200),
                                             max_suffix_len=200, pool_rows=None)
    _prefix_reuse(cfg, "sjf", 16)


def test_bf16_prefix_reuse_hpk4():
    # 32Q/8KV (hpk=4): probe batches of 32 samples = 128 rows per KV head.
    cfg = get_config("qwen3_8b_4prompts").with_(layers=2, prompt_lens=(200, 450), samples_per_prompt=36,
                                                length_dist=("lognormal", 3.5, 1.0, 1, 160), max_suffix_len=160,
                                                pool_rows=None)
    _prefix_reuse(cfg, "fptas_sjf", 8)


def test_f32_prefix_reuse_wave():
    # fp32 wavefront path: probe batches of 8 samples (16 rows).
    _prefix_reuse(get_config("tiny_f32"), "fifo", 5, split=0)


def test_bf16_single_slot_wave_prefix():
    # m=1: 2 prefix rows, so the prefix runs on the wavefront path in bf16.
    cfg = get_config("qwen3_1p7b_l1_g32").with_(slots_per_prompt=1, samples_per_prompt=4, prompt_lens=(257,),
                                                length_dist=("lognormal", 4.0, 0.8, 1, 300), max_suffix_len=300)
    _run_and_check(cfg, "fifo", capture=lambda log: sample_steps(log, every=5))


def test_response_reaches_capacity():
    # Samples of exactly max_suffix_len tokens: the last page fills completely.
    cfg = get_config("qwen3_1p7b_l1_g32").with_(samples_per_prompt=8, length_dist=("uniform", 1, 64),
                                                max_suffix_len=64)
    wl = Workload(cfg, lengths=np.array([[64, 1, 64, 17, 16, 33, 64, 2]]))
    want = oracle_log(cfg, wl, "fifo")
    _, log, steps, captured, tokens, _ = run_gpu_group(cfg, "fifo", wl=wl)
    assert log == want and np.array_equal(tokens, wl.L)
    check_against_oracle(cfg, wl, log, captured)


def test_schedule_invariance_and_determinism():
    # The output for (layer, sample, t) does not depend on the schedule or slot
    # that served it: naive and FIFO runs agree bit for bit wherever both
    # decode the same (sample, t); a repeated run is bitwise identical.
    cfg = get_config("qwen3_1p7b_g64").with_(layers=1, prompt_lens=(384,), samples_per_prompt=12,
                                             length_dist=("lognormal", 4.0, 1.0, 1, 200), max_suffix_len=200,
                                             pool_rows=None)
    runs = {}
    for name, policy in (("fifo", "fifo"), ("naive", "naive"), ("fifo2", "fifo")):
        _, log, _, captured, _, _ = run_gpu_group(cfg, policy, split=128)
        vals = {}
        for k, o in captured.items():
            for s, e in enumerate(log[k]):
                if e is not None:
                    vals[(e[1], e[2])] = o[0, s].copy()
        runs[name] = vals
    assert runs["fifo"].keys() == runs["naive"].keys()
    for key, v in runs["fifo"].items():
        assert np.array_equal(v, runs["naive"][key]), key
        assert np.array_equal(v, runs["fifo2"][key]), key


@pytest.mark.parametrize("name,every,window", [
    ("qwen3_1p7b_g64", 397, 512),      # the benchmark workload: 32 prefix rows, 16 slots
    ("longtail_g128", 997, 256),       # m=32 (64 prefix rows), responses up to 8192
    ("qwen3_8b_4prompts", 1201, 128),  # four prefixes of 256..4096, hpk=4 (64 rows per prompt), 64 slots
])
def test_full_size_sampled(name, every, window):
    # Whole workload in the launch configuration the benchmark uses; outputs of
    # sampled steps (and the first and last ones) on the first, middle and last
    # layer against the oracle.
    cfg = get_config(name)
    _run_and_check(cfg, cfg.policy, capture=lambda log: sample_steps(log, every=every, edge=2, refills=8),
                   layers=(0, cfg.layers // 2, cfg.layers - 1), window=window)


# --- softmax scale and wide score ranges ------------------------------------------------------------
# A non-default scale reaches the kernels only through infs_config.scale; inputs
# with Q scaled up and K rows ramped (qk_scale) make scores span two orders of
# magnitude, with the first prefix chunk's maximum far below later chunks' and
# the responses' (bf16 cases: about 2 against 100+, so the weight of an early
# partial underflows to exactly 0 in the online rescale and in the merge).
_BF16_SMALL = dict(layers=2, prompt_lens=(700,), samples_per_prompt=24,
                   length_dist=("lognormal", 4.0, 1.0, 1, 300), max_suffix_len=300, pool_rows=None)


@pytest.mark.parametrize("case", ["mfma32_scale1", "mfma32_wide", "mfma16_wide", "mfma64_hpk4_wide",
                                  "wave_bf16_wide", "wave_bf16_scale1"])
def test_bf16_scale_and_wide_scores(case):
    wide = (8.0, 0.1, 8.0)
    if case == "mfma32_scale1":        # 32 prefix rows on MFMA tiles, scale 1.0 at d=128
        cfg, scale = get_config("qwen3_1p7b_g64").with_(**_BF16_SMALL), 1.0
    elif case == "mfma32_wide":
        cfg, scale = get_config("qwen3_1p7b_g64").with_(**_BF16_SMALL, qk_scale=wide), 0.0
    elif case == "mfma16_wide":        # 16 rows (m=8)
        cfg, scale = get_config("qwen3_1p7b_l1_g32").with_(prompt_lens=(600,), qk_scale=wide), 0.0
    elif case == "mfma64_hpk4_wide":   # 4 query heads per KV head, 64 rows, two prompts
        cfg = get_config("qwen3_8b_4prompts").with_(layers=2, prompt_lens=(130, 511), samples_per_prompt=20,
                                                    length_dist=("lognormal", 4.0, 1.0, 1, 260),
                                                    max_suffix_len=260, pool_rows=None, qk_scale=wide)
        scale = 0.0
    else:                              # m=1: 2 prefix rows, the bf16 wavefront path
        cfg = get_config("qwen3_1p7b_l1_g32").with_(slots_per_prompt=1, samples_per_prompt=4, prompt_lens=(600,),
                                                    length_dist=("lognormal", 4.0, 0.8, 1, 300), max_suffix_len=300,
                                                    qk_scale=wide if case == "wave_bf16_wide" else None)
        scale = 1.0 if case == "wave_bf16_scale1" else 0.0
    _run_and_check(cfg, "fifo" if cfg.pred_sigma is None else "sjf", split=128,
                   capture=lambda log: sample_steps(log, every=2), scale=scale)


@pytest.mark.parametrize("case", ["scale_half", "wide"])
def test_f32_scale_and_wide_scores(case):
    # fp32 wavefront path at 1e-5, d=64, three prefix chunks of 128 tokens:
    # scale 0.5 (four times the default), or Q x 4 with K rows ramped 0.1 -> 2.
    cfg = get_config("tiny_f32").with_(prompt_lens=(300,), length_dist=("uniform", 1, 400), max_suffix_len=400)
    if case == "wide":
        cfg = cfg.with_(qk_scale=(4.0, 0.1, 2.0))
    _run_and_check(cfg, "fifo", split=128, capture=lambda log: sample_steps(log, every=3),
                   scale=0.5 if case == "scale_half" else 0.0)


def test_bf16_fixed_row_end_to_end():
    # Fixed-slot continuous sampling (Section 3.2, mode 1): slot s runs samples
    # s, s+m, s+2m, ...; step log equal to the simulator's, token counters equal
    # to the lengths, outputs against the oracle.
    cfg = get_config("qwen3_1p7b_g64").with_(**_BF16_SMALL)
    _run_and_check(cfg, "fixed_row", split=128, capture=lambda log: sample_steps(log, every=3))


def test_fp8_kv_small_every_other_step():
    # FP8 (E4M3) KV cache on the throughput workload's shape: the oracle rounds
    # every key and value to E4M3; outputs within the bf16 bound.
    cfg = get_config("qwen3_1p7b_g64").with_(layers=2, prompt_lens=(700,), samples_per_prompt=24,
                                             length_dist=("lognormal", 4.0, 1.0, 1, 300), max_suffix_len=300,
                                             pool_rows=None)
    _run_and_check(cfg, "sjf", split=128, capture=lambda log: sample_steps(log, every=2), kv_fp8=True)


def test_fp8_kv_hpk4_multi_prompt():
    cfg = get_config("qwen3_8b_4prompts").with_(layers=2, prompt_lens=(0, 130, 511), samples_per_prompt=20,
                                                length_dist=("lognormal", 4.0, 1.0, 1, 260),
                                                max_suffix_len=260, pool_rows=None)
    _run_and_check(cfg, "fptas_sjf", split=128, capture=lambda log: sample_steps(log, every=3), kv_fp8=True)


def test_fp8_kv_full_size_sampled():
    cfg = get_config("qwen3_1p7b_g64")
    _run_and_check(cfg, cfg.policy, capture=lambda log: sample_steps(log, every=397, edge=2, refills=8),
                   layers=(0, cfg.layers - 1), window=512, kv_fp8=True)
