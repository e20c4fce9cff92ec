"""Checks of the seeded input generator (CPU only)."""

import numpy as np
import torch

from workload import CONFIGS, Workload, bf16_bits_to_f64, f32_to_bf16_bits, get_config, splitmix64


def test_splitmix64_reference_outputs():
    # First three outputs of the SplitMix64 generator seeded with 0: the
    # generator adds the golden gamma before each mix, so output n is the
    # finaliser applied to n * gamma (wrapping).
    gamma = 0x9E3779B97F4A7C15
    x = np.array([0, gamma, (2 * gamma) & 0xFFFFFFFFFFFFFFFF], dtype=np.uint64)
    out = [int(v) for v in splitmix64(x)]
    assert out == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_bf16_rounding_ties_to_even():
    x = np.array([1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, -2.5, 3.0e-3], dtype=np.float32)
    bits = f32_to_bf16_bits(x)
    assert list(bits[:3]) == [0x3F80, 0x3F80, 0x3F82]


def test_bf16_rounding_matches_torch():
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32) * 3
    ours = bf16_bits_to_f64(f32_to_bf16_bits(x))
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(ours, ref)


def test_lengths_in_range_and_seeded():
    for name, cfg in CONFIGS.items():
        L = Workload.draw_lengths(cfg)
        assert L.shape == (cfg.num_prompts, cfg.samples_per_prompt)
        assert L.min() >= 1 and L.max() <= cfg.max_suffix_len
        assert np.array_equal(L, Workload.draw_lengths(cfg))


def test_dense_rows_are_unique():
    wl = Workload(get_config("tiny_f32"))
    idx = list(wl.prefix_index(0, 0))
    for i in range(8):
        idx += list(wl.suffix_index(0, 0, i, np.arange(wl.L[0, i])))
    assert len(set(idx)) == len(idx) == wl.rows_kv
    q = []
    for i in range(8):
        q += list(wl.query_index(0, 0, i, np.arange(wl.L[0, i])))
    assert sorted(q) == list(range(wl.rows_q))


def test_hashed_rows_in_pool():
    wl = Workload(get_config("qwen3_1p7b_g64"))
    idx = wl.suffix_index(27, 0, 63, np.arange(4096))
    assert idx.min() >= 0 and idx.max() < wl.rows_kv
    assert len(np.unique(idx)) > 3000
