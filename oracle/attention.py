"""Float64 decode attention over [shared prefix ; private suffix].

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper never writes the attention formula; it states the cache structure:
all G completions of a prompt reuse one prefill KV cache (Section 3.1, "KV
Cache Pooling"; Section 3.2, "Shared Prompt KV and Sample-Level Cache
Lifecycle"), and every decode step of a sample attends to the cached prompt
and its own generated tokens (Section 2.1).  The readings taken here:

* scale 1/sqrt(d) on q.k;
* grouped-query attention: query head h reads KV head floor(h / hpk),
  hpk = Hq / Hkv;
* the token decoded at this step has its K/V appended before attending, so a
  sample with t generated tokens attends to P + t keys;
* no mask beyond causality, no positional rotation (the synthetic Q/K stand
  for post-rotation activations).

This is the plain definition, with no blocking, splitting or merging: the GPU
path's split-K decomposition must reach the same numbers.
"""

import numpy as np


def default_scale(head_dim: int) -> float:
    return 1.0 / np.sqrt(float(head_dim))


def attention_weights(q: np.ndarray, k: np.ndarray, hpk: int, scale: float) -> np.ndarray:
    """Softmax weights of every query head over every key.

    q: [Hq, d]; k: [n, Hkv, d]; returns [Hq, n] (float64).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    Hq = q.shape[0]
    w = np.empty((Hq, k.shape[0]), dtype=np.float64)
    for h in range(Hq):
        g = h // hpk
        s = (k[:, g, :] @ q[h]) * scale
        e = np.exp(s - s.max())
        w[h] = e / e.sum()
    return w


def attend(q: np.ndarray, k: np.ndarray, v: np.ndarray, hpk: int, scale: float) -> np.ndarray:
    """o_h = sum_j softmax_j(scale * q_h . k_j) v_j over all n keys.

    q: [Hq, d]; k, v: [n, Hkv, d] with n >= 1; returns [Hq, d] (float64).
    """
    v = np.asarray(v, dtype=np.float64)
    w = attention_weights(q, k, hpk, scale)
    out = np.empty((w.shape[0], v.shape[2]), dtype=np.float64)
    for h in range(w.shape[0]):
        out[h] = w[h] @ v[:, h // hpk, :]
    return out


def attend_slot(wl, l: int, p: int, i: int, t: int, scale=None, kv_fp8: bool = False) -> np.ndarray:
    """Output of a live slot holding sample i of prompt p, at layer l, at the
    step where the sample's response holds t tokens (the new one included).

    Keys and values are prompt p's prefix followed by the sample's own t
    generated tokens; the values depend only on (l, p, i, t), never on which
    slot or step served them.  kv_fp8: the KV cache holds every key and value
    rounded to E4M3 (the query is not rounded).
    """
    if t < 1:
        raise ValueError("a live slot attends to at least its own new token")
    c = wl.cfg
    if scale is None:
        scale = default_scale(c.head_dim)
    kp, vp = wl.prefix_kv(l, p)
    ks, vs = wl.suffix_kv(l, p, i, t)
    k = np.concatenate([kp, ks], axis=0)
    v = np.concatenate([vp, vs], axis=0)
    if kv_fp8:
        from .fp8 import round_e4m3
        k, v = round_e4m3(k), round_e4m3(v)
    return attend(wl.query(l, p, i, t), k, v, c.hpk, scale)
