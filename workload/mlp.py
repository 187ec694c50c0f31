"""Seeded synthetic weights and inputs of a 2-layer MLP scorer (the paper
gives no trained weights, dimensions or activation; these are parameters).
No method arithmetic: only random draws and the bf16 storage rounding.

Keys: ``numpy.random.default_rng([seed, tag])``, tags 20 W1, 21 b1, 22 w2,
23 hidden states.  W1 ~ N(0, 1/Dh) stored as bf16 [H1][Dh]; b1 ~ N(0, 0.1^2);
w2 ~ N(0, 1/H1); b2 = 0; h ~ N(0, 1) bf16 [n][Dh].
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .generate import keyed_rng, to_bf16_bits

TAG_W1, TAG_B1, TAG_W2, TAG_H = 20, 21, 22, 23


@dataclass(frozen=True)
class MlpConfig:
    name: str
    seed: int
    n: int          # traces scored at once
    dim: int        # Dh
    hidden: int     # H1
    act: str        # "relu" or "gelu"


# The 512-trace workload's boundary (Qwen3-8B hidden size 4096), hidden 1024.
MLP_512 = MlpConfig(name="mlp2_512x4096_h1024_relu", seed=31, n=512, dim=4096, hidden=1024, act="relu")
# The Qwen3-32B shape (hidden size 5120), 256 traces, GELU.
MLP_256_32B = MlpConfig(name="mlp2_256x5120_h512_gelu", seed=32, n=256, dim=5120, hidden=512, act="gelu")
# Small, ragged: several tiles and a partial last tile of traces.
MLP_SMALL = MlpConfig(name="mlp2_77x256_h128_gelu", seed=33, n=77, dim=256, hidden=128, act="gelu")


def weights(cfg: MlpConfig):
    """(W1 bf16 bits [H1][Dh], b1 f32 [H1], w2 f32 [H1], b2)."""
    W1 = keyed_rng(cfg.seed, TAG_W1).standard_normal((cfg.hidden, cfg.dim), dtype=np.float32) / np.float32(np.sqrt(cfg.dim))
    b1 = (keyed_rng(cfg.seed, TAG_B1).standard_normal(cfg.hidden, dtype=np.float32) * np.float32(0.1)).astype(np.float32)
    w2 = (keyed_rng(cfg.seed, TAG_W2).standard_normal(cfg.hidden, dtype=np.float32) / np.float32(np.sqrt(cfg.hidden))).astype(np.float32)
    return to_bf16_bits(W1), b1, w2, 0.0


def hidden_states(cfg: MlpConfig, n: int | None = None) -> np.ndarray:
    n = cfg.n if n is None else n
    return to_bf16_bits(keyed_rng(cfg.seed, TAG_H).standard_normal((n, cfg.dim), dtype=np.float32))
