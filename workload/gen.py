"""Seeded draws for one group-decode workload.

Three independent random streams per workload, seeded from the preset's
``seed`` k:

* lengths:      PCG64(1000 + k) -- true completion length L of every sample;
* prediction:   PCG64(2000 + k) -- predicted length L_hat = L * exp(N(0, s^2));
* Q/K/V pools:  PCG64([3000 + k, kind]) -- i.i.d. N(0, 1) rows, rounded to the
                storage type (bf16 round-to-nearest-even, or kept fp32).

A decode row is addressed by (layer l, prompt p, sample i, position t).  Small
workloads give every row its own pool entry ("dense" indexing, so all values
are i.i.d.).  Large workloads draw a fixed pool of R rows and map each address
to ``splitmix64(seed ^ key) mod R`` -- SplitMix64 is the integer mixer of
Steele, Lea and Flood (OOPSLA 2014) -- so any row can be regenerated in O(1)
without materialising tens of GB of activations.  Prefix rows use the same
scheme with their own key tag.

Nothing here computes attention or schedules slots.
"""

import numpy as np

from .configs import GroupConfig

_MASK64 = np.uint64(0xFFFFFFFFFFFFFFFF)

TAG_PREFIX = 1
TAG_SUFFIX = 2
TAG_QUERY = 3


def splitmix64(x):
    """SplitMix64 finaliser on a uint64 array (wrap-around arithmetic)."""
    z = np.asarray(x, dtype=np.uint64) + np.uint64(0x9E3779B97F4A7C15)
    z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
    z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
    return z ^ (z >> np.uint64(31))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (round to nearest, ties to even); returns uint16 bits.

    Inputs here are finite normal draws, so no NaN handling is needed.
    """
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (b >> np.uint32(16)) & np.uint32(1)
    r = (b + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of bf16 bit patterns as float64."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def _key(tag, l, p, i, t):
    """Pack a row address into 64 bits: tag:4 | l:12 | p:8 | i:16 | t:24."""
    t = np.asarray(t, dtype=np.uint64)
    return (np.uint64(tag) << np.uint64(60)) | (np.uint64(l) << np.uint64(48)) | \
           (np.uint64(p) << np.uint64(40)) | (np.uint64(i) << np.uint64(24)) | t


class Workload:
    """Lengths, predicted lengths and Q/K/V row pools of one preset."""

    def __init__(self, cfg: GroupConfig, lengths=None, pred=None):
        self.cfg = cfg
        if lengths is None:
            lengths = self.draw_lengths(cfg)
        self.L = np.asarray(lengths, dtype=np.int32).reshape(cfg.num_prompts, cfg.samples_per_prompt)
        if pred is None:
            pred = self.draw_predictions(cfg, self.L)
        self.L_hat = np.asarray(pred, dtype=np.float64).reshape(self.L.shape)
        if int(self.L.min()) < 1 or int(self.L.max()) > cfg.max_suffix_len:
            raise ValueError("lengths must lie in [1, max_suffix_len]")
        self._cumL = np.concatenate([[0], np.cumsum(self.L.reshape(-1).astype(np.int64))])
        self._cumP = np.concatenate([[0], np.cumsum(np.asarray(cfg.prompt_lens, dtype=np.int64))])
        self.dense = cfg.pool_rows is None
        if self.dense:
            tot_suffix = int(self._cumL[-1])
            self.rows_q = cfg.layers * tot_suffix
            self.rows_kv = cfg.layers * (int(self._cumP[-1]) + tot_suffix)
        else:
            self.rows_q = self.rows_kv = int(cfg.pool_rows)
        self._pools = {}

    # ---------------------------------------------------------------- lengths
    @staticmethod
    def draw_lengths(cfg: GroupConfig) -> np.ndarray:
        rng = np.random.Generator(np.random.PCG64(1000 + cfg.seed))
        n = cfg.samples_per_prompt
        out = []
        for _ in range(cfg.num_prompts):
            kind = cfg.length_dist[0]
            if kind == "uniform":
                _, lo, hi = cfg.length_dist
                L = rng.integers(lo, hi, size=n, endpoint=True)
            elif kind == "lognormal":
                _, mu, sigma, lo, hi = cfg.length_dist
                L = np.clip(np.rint(np.exp(rng.normal(mu, sigma, size=n))), lo, hi)
            elif kind == "mixture":
                _, p_long, mu, sigma, lo, hi, ulo, uhi = cfg.length_dist
                pick = rng.random(size=n) < p_long
                ln = np.clip(np.rint(np.exp(rng.normal(mu, sigma, size=n))), lo, hi)
                un = rng.integers(ulo, uhi, size=n, endpoint=True)
                L = np.where(pick, un, ln)
            else:
                raise ValueError(f"unknown length distribution {kind!r}")
            out.append(np.asarray(L, dtype=np.int32))
        return np.stack(out)

    @staticmethod
    def draw_predictions(cfg: GroupConfig, L: np.ndarray) -> np.ndarray:
        if cfg.pred_sigma is None:
            return L.astype(np.float64)
        rng = np.random.Generator(np.random.PCG64(2000 + cfg.seed))
        noise = np.exp(rng.normal(0.0, cfg.pred_sigma, size=L.shape))
        return L.astype(np.float64) * noise

    # ------------------------------------------------------------------ pools
    def _shape(self, kind):
        c = self.cfg
        heads = c.num_q_heads if kind == "q" else c.num_kv_heads
        rows = self.rows_q if kind == "q" else self.rows_kv
        return rows, heads, c.head_dim

    def pool(self, kind: str) -> np.ndarray:
        """Stored values of one pool ('q', 'k' or 'v'): uint16 bf16 bits or float32."""
        if kind not in self._pools:
            stream = {"q": 0, "k": 1, "v": 2}[kind]
            rng = np.random.Generator(np.random.PCG64([3000 + self.cfg.seed, stream]))
            x = rng.standard_normal(self._shape(kind), dtype=np.float32)
            if self.cfg.qk_scale is not None:
                q_scale, k_first, k_last = self.cfg.qk_scale
                if kind == "q":
                    x *= np.float32(q_scale)
                elif kind == "k":
                    x *= np.linspace(k_first, k_last, x.shape[0], dtype=np.float32)[:, None, None]
            self._pools[kind] = f32_to_bf16_bits(x) if self.cfg.dtype == "bf16" else x
        return self._pools[kind]

    def values(self, kind: str, idx) -> np.ndarray:
        """Exact stored values of pool rows ``idx`` as float64, shape [n, H, d]."""
        rows = self.pool(kind)[np.asarray(idx, dtype=np.int64)]
        return bf16_bits_to_f64(rows) if self.cfg.dtype == "bf16" else rows.astype(np.float64)

    # ---------------------------------------------------------------- indexing
    def _hashed(self, tag, l, p, i, t):
        seed = np.uint64((0xD1B54A32D192ED03 * (3000 + self.cfg.seed)) & 0xFFFFFFFFFFFFFFFF)
        h = splitmix64(_key(tag, l, p, i, t) ^ seed)
        return (h % np.uint64(self.rows_kv if tag != TAG_QUERY else self.rows_q)).astype(np.int64)

    def prefix_index(self, l: int, p: int) -> np.ndarray:
        """K/V pool rows of prompt p's prefix tokens 0..P_p-1 at layer l."""
        P = self.cfg.prompt_lens[p]
        j = np.arange(P, dtype=np.int64)
        if self.dense:
            return l * int(self._cumP[-1]) + int(self._cumP[p]) + j
        return self._hashed(TAG_PREFIX, l, p, 0, j)

    def suffix_index(self, l: int, p: int, i: int, t) -> np.ndarray:
        """K/V pool rows of sample (p, i)'s generated tokens at positions t."""
        t = np.asarray(t, dtype=np.int64)
        if self.dense:
            c = self.cfg
            flat = p * c.samples_per_prompt + i
            base = c.layers * int(self._cumP[-1]) + l * int(self._cumL[-1]) + int(self._cumL[flat])
            return base + t
        return self._hashed(TAG_SUFFIX, l, p, i, t)

    def query_index(self, l: int, p: int, i: int, t) -> np.ndarray:
        """Q pool rows of sample (p, i)'s query at positions t (suffix length t+1)."""
        t = np.asarray(t, dtype=np.int64)
        if self.dense:
            flat = p * self.cfg.samples_per_prompt + i
            return l * int(self._cumL[-1]) + int(self._cumL[flat]) + t
        return self._hashed(TAG_QUERY, l, p, i, t)

    # ------------------------------------------------------------ conveniences
    def prefix_kv(self, l: int, p: int):
        """(K, V) of prompt p's prefix at layer l, float64 [P, Hkv, d]."""
        idx = self.prefix_index(l, p)
        return self.values("k", idx), self.values("v", idx)

    def suffix_kv(self, l: int, p: int, i: int, t: int):
        """(K, V) of sample (p, i)'s first t generated tokens at layer l, float64 [t, Hkv, d]."""
        idx = self.suffix_index(l, p, i, np.arange(t))
        return self.values("k", idx), self.values("v", idx)

    def query(self, l: int, p: int, i: int, t: int) -> np.ndarray:
        """Query of sample (p, i) when its suffix holds t tokens (t >= 1), float64 [Hq, d]."""
        return self.values("q", self.query_index(l, p, i, [t - 1]))[0]

    @property
    def total_tokens(self) -> int:
        return int(self.L.sum())


# Length settings of the scheduler comparison: completion lengths
# clip(rint(exp(N(mu, sigma))), 1, cap), with means of a few hundred tokens at a
# 1024-token cap as in the paper's experiments (Section 5.1).  They stand in for
# the datasets' real completion lengths, which are not used.
SCHEDULER_STUDY = (
    ("short (mean ~180)", 4.95, 0.75),
    ("medium (mean ~420)", 5.85, 0.8),
    ("long (mean ~610)", 6.35, 0.9),
)


def scheduler_study_lengths(mu, sigma, n_groups, G, cap=1024, pred_sigma=0.2, seed=0):
    """n_groups independent groups of G true lengths and their predictions
    L * exp(N(0, pred_sigma^2)); PCG64(5000 + seed) and PCG64(6000 + seed)."""
    rng = np.random.Generator(np.random.PCG64(5000 + seed))
    L = np.clip(np.rint(np.exp(rng.normal(mu, sigma, size=(n_groups, G)))), 1, cap).astype(np.int32)
    noise = np.random.Generator(np.random.PCG64(6000 + seed)).normal(0.0, pred_sigma, size=L.shape)
    return L, L.astype(np.float64) * np.exp(noise)


def scheduler_study_stream(mu, sigma, L, extra, cap=1024, seed=0):
    """Per group, a dynamic-slot stream: the group's own lengths L[n] followed
    by `extra` more draws of the same distribution (PCG64(7000 + seed))."""
    rng = np.random.Generator(np.random.PCG64(7000 + seed))
    more = np.clip(np.rint(np.exp(rng.normal(mu, sigma, size=(L.shape[0], extra)))), 1, cap).astype(np.int32)
    return np.concatenate([L, more], axis=1)
