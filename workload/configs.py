"""Named group-decode workloads.

Each preset fixes the model shape (attention path only), the shared prompt
lengths, the group size G, the number of live slots m per prompt, the
completion-length distribution and the refill policy.  The shapes follow the
Qwen3-1.7B / Qwen3-8B attention layout (16 or 32 query heads, 8 KV heads,
head_dim 128); the defaults of the paper's experiments (G=32, g=4, at most
1024 generated tokens) are described in its Section 5.1.  The synthetic
lognormal lengths stand in for the real completion lengths of the paper's
datasets, and ``L * lognormal(0, 0.2)`` stands in for the BERT length
predictor of Section 4.
"""

from dataclasses import dataclass, field, replace
from typing import Optional, Tuple


@dataclass(frozen=True)
class GroupConfig:
    name: str
    layers: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    prompt_lens: Tuple[int, ...]
    samples_per_prompt: int          # G
    slots_per_prompt: int            # m (the paper's micro-group size g)
    length_dist: Tuple               # see Workload.draw_lengths
    max_suffix_len: int
    policy: str                      # refill policy timed for this workload
    pred_sigma: Optional[float]      # sigma of the multiplicative prediction noise
    dtype: str                       # "f32" or "bf16": storage type of Q, K, V
    seed: int
    pool_rows: Optional[int] = None  # None: every (layer, prompt, sample, t) row is unique
    description: str = ""
    # Wide score ranges: (q_scale, k_first, k_last) multiplies every Q draw by
    # q_scale and K pool row r by a factor rising linearly from k_first (row 0)
    # to k_last (last row), before rounding to the storage type.  Rows are laid
    # out prefix first (token order), then responses, so later prefix chunks and
    # the responses reach much larger scores than the first prefix chunk.
    qk_scale: Optional[Tuple[float, float, float]] = None

    @property
    def num_prompts(self) -> int:
        return len(self.prompt_lens)

    @property
    def hpk(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def num_slots(self) -> int:
        return self.num_prompts * self.slots_per_prompt

    @property
    def prefix_rows(self) -> int:
        """Query rows that share one KV head of one prompt's prefix: m * hpk."""
        return self.slots_per_prompt * self.hpk

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def with_(self, **kw) -> "GroupConfig":
        return replace(self, **kw)


CONFIGS = {
    # 1 layer, GQA 4/2, d=64, P=32, G=8, m=4, lengths U[1,64], fp32.
    "tiny_f32": GroupConfig(
        name="tiny_f32", layers=1, num_q_heads=4, num_kv_heads=2, head_dim=64,
        prompt_lens=(32,), samples_per_prompt=8, slots_per_prompt=4,
        length_dist=("uniform", 1, 64), max_suffix_len=64, policy="fifo",
        pred_sigma=None, dtype="f32", seed=1,
        description="1 layer, 4Q/2KV heads, d=64, prompt 32, G=8, m=4, L~U[1,64], fp32"),
    # Qwen3-1.7B-shaped single layer.
    "qwen3_1p7b_l1_g32": GroupConfig(
        name="qwen3_1p7b_l1_g32", layers=1, num_q_heads=16, num_kv_heads=8, head_dim=128,
        prompt_lens=(512,), samples_per_prompt=32, slots_per_prompt=8,
        length_dist=("lognormal", 6.0, 0.8, 16, 2048), max_suffix_len=2048, policy="fifo",
        pred_sigma=None, dtype="bf16", seed=2,
        description="1 layer, 16Q/8KV, d=128, prompt 512, G=32, m=8, L~LN(6,0.8) in [16,2048], bf16"),
    # Qwen3-1.7B-shaped, 28 layers: the throughput workload.
    "qwen3_1p7b_g64": GroupConfig(
        name="qwen3_1p7b_g64", layers=28, num_q_heads=16, num_kv_heads=8, head_dim=128,
        prompt_lens=(2048,), samples_per_prompt=64, slots_per_prompt=16,
        length_dist=("lognormal", 6.5, 1.0, 32, 4096), max_suffix_len=4096, policy="sjf",
        pred_sigma=0.2, dtype="bf16", seed=3, pool_rows=1 << 15,
        description="28 layers, 16Q/8KV, d=128, prompt 2048, G=64, m=16, L~LN(6.5,1) in [32,4096], SJF, bf16"),
    # Long-tail group.
    "longtail_g128": GroupConfig(
        name="longtail_g128", layers=28, num_q_heads=16, num_kv_heads=8, head_dim=128,
        prompt_lens=(1024,), samples_per_prompt=128, slots_per_prompt=32,
        length_dist=("mixture", 0.2, 6.0, 0.7, 1, 8192, 4096, 8192), max_suffix_len=8192,
        policy="sjf", pred_sigma=0.2, dtype="bf16", seed=4, pool_rows=1 << 15,
        description="28 layers, 16Q/8KV, d=128, prompt 1024, G=128, m=32, "
                    "80% LN(6,0.7) + 20% U[4096,8192], SJF, bf16"),
    # Qwen3-8B-shaped, four prompts decoded in one batch.
    "qwen3_8b_4prompts": GroupConfig(
        name="qwen3_8b_4prompts", layers=36, num_q_heads=32, num_kv_heads=8, head_dim=128,
        prompt_lens=(256, 1024, 2048, 4096), samples_per_prompt=64, slots_per_prompt=16,
        length_dist=("lognormal", 6.5, 1.0, 16, 8192), max_suffix_len=8192, policy="sjf",
        pred_sigma=0.2, dtype="bf16", seed=5, pool_rows=1 << 14,
        description="36 layers, 32Q/8KV, d=128, prompts 256/1024/2048/4096, G=64 each, "
                    "m=16 each, L~LN(6.5,1) in [16,8192], SJF, bf16"),
}

BENCH_CONFIG = "qwen3_1p7b_g64"


def get_config(name: str, **overrides) -> GroupConfig:
    cfg = CONFIGS[name]
    return cfg.with_(**overrides) if overrides else cfg
