"""Workload shapes for the PASK decode hot path.

Five workloads, from a tiny case that a pure-Python check finishes in seconds
to a Qwen3-32B-shaped attention at serving batch.  The model geometries are
those of the models the paper evaluates (Qwen3-4B-Instruct; Section 4.1) and
of a larger GQA model; weights are never used, only the attention shapes.
"""

from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Tuple


@dataclass(frozen=True)
class Config:
    name: str
    batch: int
    n_layers: int
    n_groups: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    prompt_min: int
    prompt_max: int
    prompt_dist: str          # "fixed" | "uniform" | "loguniform"
    gen_tokens: int
    tag_source: str           # "iid" | "calls" (tool-call output read by the tagger)
    prompt_tagged: bool       # prompt KV governed by the table (prompt-side companion)
    budgets: Tuple[float, ...]
    n_sink: int
    seed: int
    page_tokens: int = 16
    resident_layers: int = 0  # 0: all layers resident; else only this many (one GPU's share)
    notes: str = field(default="", compare=False)

    @property
    def group_size(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def layers_resident(self) -> int:
        return self.resident_layers or self.n_layers

    @property
    def n_tags(self) -> int:
        return 12 if self.prompt_tagged else 6

    def with_budget(self, beta: float) -> "Config":
        return replace(self, budgets=(beta,))


CONFIGS = [
    Config(
        name="tiny_b1_l2_h8x2_d64",
        batch=1, n_layers=2, n_groups=2, n_q_heads=8, n_kv_heads=2, head_dim=64,
        prompt_min=256, prompt_max=256, prompt_dist="fixed",
        gen_tokens=128, tag_source="iid", prompt_tagged=False,
        budgets=(0.33,), n_sink=0, seed=1000,
        notes="parity-only; tags i.i.d. uniform over the 6 decode tags",
    ),
    Config(
        name="qwen3_4b_b1_p2048_g512",
        batch=1, n_layers=36, n_groups=4, n_q_heads=32, n_kv_heads=8, head_dim=128,
        prompt_min=2048, prompt_max=2048, prompt_dist="fixed",
        gen_tokens=512, tag_source="calls", prompt_tagged=False,
        budgets=(0.33,), n_sink=0, seed=1001,
    ),
    Config(
        name="qwen3_4b_b64_p1k-8k_g1024",
        batch=64, n_layers=36, n_groups=4, n_q_heads=32, n_kv_heads=8, head_dim=128,
        prompt_min=1024, prompt_max=8192, prompt_dist="uniform",
        gen_tokens=1024, tag_source="calls", prompt_tagged=False,
        budgets=(0.33,), n_sink=0, seed=1002,
    ),
    Config(
        name="qwen3_4b_b128_p4k-16k_tagged_g512",
        batch=128, n_layers=36, n_groups=4, n_q_heads=32, n_kv_heads=8, head_dim=128,
        prompt_min=4096, prompt_max=16384, prompt_dist="uniform",
        gen_tokens=512, tag_source="calls", prompt_tagged=True,
        budgets=(0.25, 0.33, 0.5, 1.0), n_sink=16, seed=1003,
    ),
    Config(
        name="qwen3_32b_attn_b256_p16k-32k_g2048",
        batch=256, n_layers=64, n_groups=8, n_q_heads=64, n_kv_heads=8, head_dim=128,
        prompt_min=16384, prompt_max=32768, prompt_dist="loguniform",
        gen_tokens=2048, tag_source="calls", prompt_tagged=False,
        budgets=(0.33,), n_sink=0, seed=1004, resident_layers=8,
        notes="one layer group (8 layers) resident: one GPU's share of a 64-layer cache",
    ),
]


def get_config(i: int) -> Config:
    return CONFIGS[i]
