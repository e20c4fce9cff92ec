"""Seeded random small workloads on the GPU against the float64 oracle:
element type, head size, heads per KV head, slots, prompts (lengths 0, 1 and
around the 32-token block and 128-token chunk edges), samples, split-K chunk
length, refill policy and the E4M3 cache are drawn per case; every other step
is compared (bf16 / E4M3 within 1e-2, fp32 within 1e-5), the step log and the
token counters bit-exactly."""

import numpy as np
import pytest

from tests.gpu_harness import check_against_oracle, oracle_log, run_gpu_group, say
from workload import Workload, get_config

pytestmark = pytest.mark.gpu

PROMPT_LENS = (0, 1, 17, 31, 32, 33, 127, 128, 129, 300)
POLICIES = ("naive", "fifo", "sjf", "fptas_sjf", "lpt")


def draw_case(seed):
    rng = np.random.default_rng(1000 + seed)
    bf16 = bool(rng.integers(0, 2))
    d = int(rng.choice([64, 128], p=[0.3, 0.7]))
    hpk = int(rng.choice([1, 2, 4, 8]))
    NP = int(rng.integers(1, 4))
    max_rows = 128 if bf16 else 16
    m_max = max(1, min(64 // NP, max_rows // hpk))
    m = int(rng.integers(1, m_max + 1))
    kv8 = bf16 and d == 128 and m * hpk >= 16 and bool(rng.integers(0, 2))
    prompts = tuple(int(x) for x in rng.choice(PROMPT_LENS, NP))
    G = int(rng.integers(1, 2 * m + 4))
    top = int(rng.choice([20, 80, 300]))
    split = int(rng.choice([0, 128]))
    policy = str(rng.choice(POLICIES))
    cfg = get_config("tiny_f32").with_(
        name=f"random_{seed}", layers=int(rng.integers(1, 3)), num_q_heads=2 * hpk, num_kv_heads=2, head_dim=d,
        prompt_lens=prompts, samples_per_prompt=G, slots_per_prompt=m, length_dist=("uniform", 1, top),
        max_suffix_len=top, dtype="bf16" if bf16 else "f32", pred_sigma=0.3, seed=2000 + seed)
    return cfg, policy, split, kv8


@pytest.mark.parametrize("seed", range(24))
def test_random_small_workload(seed):
    cfg, policy, split, kv8 = draw_case(seed)
    wl = Workload(cfg)
    want = oracle_log(cfg, wl, policy)
    _, log, steps, captured, tokens, _ = run_gpu_group(cfg, policy, wl=wl, split=split, kv_fp8=kv8,
                                                       capture=lambda k: k % 2 == 0 or k == len(want) - 1)
    assert log == want and steps == len(want)
    assert np.array_equal(tokens, wl.L)
    worst, n = check_against_oracle(cfg, wl, log, captured, kv_fp8=kv8)
    say(f"  [{cfg.name}: {cfg.dtype} d={cfg.head_dim} hpk={cfg.hpk} m={cfg.slots_per_prompt} P={cfg.prompt_lens} "
        f"G={cfg.samples_per_prompt} L<={cfg.max_suffix_len} split={split or 256} {policy}{' e4m3' if kv8 else ''}] "
        f"{steps} steps, {n} outputs, max abs err {worst:.3g}")
