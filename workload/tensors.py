"""Seeded bf16 tensors and prompt lengths.

Q, K and V entries are drawn N(0, 1) in fp32 from a seeded torch generator
and rounded to bf16 (torch's conversion is round-to-nearest-even).  Sub-seeds
are derived with numpy's SeedSequence keyed by purpose, layer and sequence, so
any single (layer, sequence) slice can be regenerated on its own.
"""

from __future__ import annotations

import numpy as np
import torch

PURPOSE = {"prompt_k": 1, "prompt_v": 2, "gen_k": 3, "gen_v": 4, "q": 5,
           "tags": 6, "lengths": 7, "policy": 8, "outlier": 9, "prompt_tags": 10, "device_inputs": 11}


def sub_seed(seed: int, purpose: str, *keys: int) -> int:
    ss = np.random.SeedSequence([int(seed), PURPOSE[purpose], *[int(k) for k in keys]])
    return int(ss.generate_state(1, dtype=np.uint64)[0] & ((1 << 63) - 1))


def bf16_normal(shape, seed: int, device="cpu", outlier_channels: int = 0,
                outlier_scale: float = 8.0) -> torch.Tensor:
    """N(0,1) in fp32 -> bf16 (RNE).  Optionally scale a few random channels of
    the last axis (outlier channels) to stress the group quantiser."""
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if outlier_channels:
        rng = np.random.default_rng(seed ^ 0x5EED)
        ch = rng.choice(shape[-1], size=outlier_channels, replace=False)
        x[..., torch.as_tensor(ch, device=device)] *= outlier_scale
    return x.to(torch.bfloat16)


def prompt_lengths(cfg, seed: int | None = None) -> np.ndarray:
    """Per-sequence prompt lengths for a workload."""
    seed = cfg.seed if seed is None else seed
    rng = np.random.default_rng(sub_seed(seed, "lengths"))
    if cfg.prompt_dist == "fixed":
        return np.full(cfg.batch, cfg.prompt_min, dtype=np.int64)
    if cfg.prompt_dist == "uniform":
        return rng.integers(cfg.prompt_min, cfg.prompt_max + 1, size=cfg.batch).astype(np.int64)
    if cfg.prompt_dist == "loguniform":
        u = rng.uniform(np.log(cfg.prompt_min), np.log(cfg.prompt_max), size=cfg.batch)
        return np.round(np.exp(u)).astype(np.int64)
    raise ValueError(cfg.prompt_dist)
