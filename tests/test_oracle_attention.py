"""Pins for the float64 attention oracle (CPU only).

Each check ties the oracle to something other than itself: closed forms of
softmax attention, torch's scaled_dot_product_attention over a physically
duplicated prefix, invariants, and pure-Python brute force.
"""

import math

import numpy as np
import pytest
import torch

from oracle import attend, attend_slot, attention_weights, default_scale, simulate
from workload import Workload, get_config
from tests.brute import brute_attend_slot


def _rand(rng, *shape):
    return rng.standard_normal(shape)


def test_closed_form_three_quarters():
    # d = 2, scale 1/sqrt(2): q.k0 * scale = ln 3 and q.k1 = 0, so the two
    # weights are 3/4 and 1/4, and o = 3/4 v0 + 1/4 v1.
    q = np.array([[math.sqrt(2.0) * math.log(3.0), 0.0]])
    k = np.array([[[1.0, 0.0]], [[0.0, 0.0]]])
    v = np.array([[[1.0, 0.0]], [[0.0, 1.0]]])
    w = attention_weights(q, k, 1, default_scale(2))
    assert np.allclose(w, [[0.75, 0.25]], atol=1e-15)
    assert np.allclose(attend(q, k, v, 1, default_scale(2)), [[0.75, 0.25]], atol=1e-15)


def test_equal_keys_give_mean_of_values():
    rng = np.random.default_rng(0)
    n, Hkv, hpk, d = 37, 2, 3, 16
    k = np.broadcast_to(_rand(rng, 1, Hkv, d), (n, Hkv, d)).copy()
    v = _rand(rng, n, Hkv, d)
    q = _rand(rng, Hkv * hpk, d)
    o = attend(q, k, v, hpk, 0.25)
    for h in range(Hkv * hpk):
        assert np.allclose(o[h], v[:, h // hpk].mean(axis=0), atol=1e-13)


def test_equal_values_give_that_value():
    rng = np.random.default_rng(1)
    n, Hkv, hpk, d = 29, 2, 2, 8
    c = _rand(rng, Hkv, d)
    v = np.broadcast_to(c, (n, Hkv, d)).copy()
    o = attend(_rand(rng, Hkv * hpk, d), _rand(rng, n, Hkv, d), v, hpk, 0.3)
    for h in range(Hkv * hpk):
        assert np.allclose(o[h], c[h // hpk], atol=1e-13)


def test_gqa_head_map_against_per_head_mha():
    # hpk = 1 is plain multi-head attention; query head h of a GQA layer must
    # equal MHA on KV head floor(h / hpk) (not h mod Hkv).
    rng = np.random.default_rng(2)
    n, Hkv, hpk, d = 11, 3, 4, 8
    q, k, v = _rand(rng, Hkv * hpk, d), _rand(rng, n, Hkv, d), _rand(rng, n, Hkv, d)
    o = attend(q, k, v, hpk, 0.5)
    for h in range(Hkv * hpk):
        g = h // hpk
        o1 = attend(q[h:h + 1], k[:, g:g + 1], v[:, g:g + 1], 1, 0.5)
        assert np.allclose(o[h], o1[0], atol=1e-14)


def test_weights_nonnegative_and_sum_to_one():
    rng = np.random.default_rng(3)
    w = attention_weights(_rand(rng, 8, 32) * 4, _rand(rng, 300, 2, 32) * 4, 4, default_scale(32))
    assert (w >= 0).all()
    assert np.allclose(w.sum(axis=1), 1.0, atol=1e-12)


def test_key_permutation_invariance():
    rng = np.random.default_rng(4)
    q, k, v = _rand(rng, 4, 16), _rand(rng, 50, 2, 16), _rand(rng, 50, 2, 16)
    perm = rng.permutation(50)
    assert np.allclose(attend(q, k, v, 2, 0.25), attend(q, k[perm], v[perm], 2, 0.25), atol=1e-13)


def test_split_merge_equals_unsplit():
    # Softmax over a union of key sets equals the log-sum-exp combination of
    # the softmaxes over the parts -- the identity a split-K kernel relies on.
    rng = np.random.default_rng(5)
    q, k, v = _rand(rng, 2, 8), _rand(rng, 40, 1, 8), _rand(rng, 40, 1, 8)
    full = attend(q, k, v, 2, 0.4)
    cuts = [0, 7, 8, 25, 40]
    for h in range(2):
        ms, ls, os_ = [], [], []
        for a, b in zip(cuts[:-1], cuts[1:]):
            s = k[a:b, 0] @ q[h] * 0.4
            mx = s.max()
            e = np.exp(s - mx)
            ms.append(mx), ls.append(e.sum()), os_.append(e @ v[a:b, 0])
        M = max(ms)
        num = sum(math.exp(mk - M) * ok for mk, ok in zip(ms, os_))
        den = sum(math.exp(mk - M) * lk for mk, lk in zip(ms, ls))
        assert np.allclose(num / den, full[h], atol=1e-13)


@pytest.mark.parametrize("name", ["tiny_f32", "qwen3_1p7b_l1_g32"])
def test_decomposition_equals_sdpa_over_duplicated_prefix(name):
    # North-star check 1: the shared-prefix output equals torch's SDPA (float64,
    # CPU) when every slot physically carries its own copy of the prefix and
    # the KV heads are repeated hpk times.
    cfg = get_config(name)
    if name != "tiny_f32":
        cfg = cfg.with_(prompt_lens=(64,), samples_per_prompt=4)
    wl = Workload(cfg)
    hpk = cfg.hpk
    for i in range(cfg.samples_per_prompt):
        t = int(min(wl.L[0, i], 23))
        kp, vp = wl.prefix_kv(0, 0)
        ks, vs = wl.suffix_kv(0, 0, i, t)
        k = torch.from_numpy(np.concatenate([kp.copy(), ks])).permute(1, 0, 2)    # [Hkv, n, d]
        v = torch.from_numpy(np.concatenate([vp.copy(), vs])).permute(1, 0, 2)
        k = k.repeat_interleave(hpk, dim=0)[None]
        v = v.repeat_interleave(hpk, dim=0)[None]
        q = torch.from_numpy(wl.query(0, 0, i, t))[None, :, None, :]
        ref = torch.nn.functional.scaled_dot_product_attention(q, k, v)[0, :, 0, :].numpy()
        assert np.allclose(attend_slot(wl, 0, 0, i, t), ref, atol=1e-12, rtol=0)


def test_brute_force_tiny():
    # North-star check 3 (attention part): pure-Python fsum brute force.
    cfg = get_config("tiny_f32").with_(head_dim=8, prompt_lens=(5,), length_dist=("uniform", 1, 12),
                                       max_suffix_len=12)
    wl = Workload(cfg)
    for i in (0, 3, 7):
        for t in sorted({1, int(wl.L[0, i]) // 2 + 1, int(wl.L[0, i])}):
            o = attend_slot(wl, 0, 0, i, t)
            for h in range(cfg.num_q_heads):
                assert np.allclose(o[h], brute_attend_slot(wl, 0, 0, i, t, h), atol=1e-12, rtol=0)


def test_empty_prefix_is_plain_causal_decode():
    # P = 0: the slot attends to its own tokens only; equals attend() over
    # the suffix rows alone.
    cfg = get_config("tiny_f32").with_(prompt_lens=(0,))
    wl = Workload(cfg)
    ks, vs = wl.suffix_kv(0, 0, 2, 5)
    ref = attend(wl.query(0, 0, 2, 5), ks, vs, cfg.hpk, default_scale(cfg.head_dim))
    assert np.allclose(attend_slot(wl, 0, 0, 2, 5), ref, atol=0)


def test_schedule_invariance_of_values():
    # The output for (layer, sample, t) depends only on those, so every
    # policy's step log maps to the same values for a given (sample, t).
    cfg = get_config("tiny_f32")
    wl = Workload(cfg)
    seen = {}
    for policy in ("naive", "fifo", "fixed_row"):
        r = simulate(wl.L[0], cfg.slots_per_prompt, policy)
        for row in r.log[::5]:
            for e in row:
                if e is None:
                    continue
                i, t = e
                o = attend_slot(wl, 0, 0, i, t)
                if (i, t) in seen:
                    assert np.array_equal(seen[(i, t)], o)
                seen[(i, t)] = o


def test_large_scores_stay_finite():
    # Scores near 1e3 overflow exp() unless the row maximum is subtracted
    # first; the exact answer here is the value row of the largest score.
    q = np.array([[40.0, 0.0, 0.0, 0.0]])
    k = np.array([[[50.0, 0, 0, 0]], [[-50.0, 0, 0, 0]], [[49.0, 0, 0, 0]]])
    v = np.array([[[1.0, 2, 3, 4]], [[5.0, 6, 7, 8]], [[9.0, 9, 9, 9]]])
    o = attend(q, k, v, 1, 1.0)
    assert np.isfinite(o).all()
    # weights: e^0 : e^-4000 : e^-40  -> the third is e^-40 relative.
    w3 = math.exp(-40.0) / (1 + math.exp(-40.0))
    assert np.allclose(o[0], (1 - w3) * v[0, 0] + w3 * v[2, 0], atol=1e-15)
