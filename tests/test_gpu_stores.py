"""GPU: the prefix store and the response pages hold exactly the K/V rows they
were given (read back through the C ABI, compared bit for bit), for the plain
and the MFMA-swizzled prefix layouts and for pages written by the append."""

import numpy as np
import pytest

from tests.gpu_harness import run_gpu_group, say
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
