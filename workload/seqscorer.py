"""Seeded synthetic weights and step states of a history-aware sequence
scorer (App. A.1, Eqs. 4-6: input LN, W_in, GELU, causal Transformer layers
with RoPE and SwiGLU, output LN, w_out, sigmoid).  The paper gives no widths,
depth, head count or trained weights: they are parameters here.  No method
arithmetic: only random draws and storage rounding (weights fp32, step
states bf16).

Keys: ``numpy.random.default_rng([seed, tag, *ids])``: tag 40 input LN,
41 W_in, 42 layer l's weights (ids l, k for its k-th tensor), 43 output LN
and w_out, 44 step states (id: round).  Linear weights ~ N(0, 1/fan_in); LN
gains 1 + N(0, 0.1^2), LN biases N(0, 0.1^2); step states N(0, 1).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .generate import keyed_rng, to_bf16_bits

TAG_LN_IN, TAG_WIN, TAG_LAYER, TAG_OUT, TAG_H = 40, 41, 42, 43, 44


@dataclass(frozen=True)
class SeqScorerConfig:
    name: str
    seed: int
    input_dim: int     # D, the LLM hidden size
    d_model: int
    n_heads: int
    n_layers: int
    d_ff: int          # SwiGLU hidden width
    max_steps: int     # step states a trace can hold
    slots: int         # trace slots


# Small, for every-step parity: two layers, two heads, ragged trace counts.
SEQ_SMALL = SeqScorerConfig(name="seqscorer_d128_l2_small", seed=41, input_dim=256, d_model=128, n_heads=2,
                            n_layers=2, d_ff=256, max_steps=40, slots=24)
# The 512-trace workload's boundary (Qwen3-8B hidden size 4096).
SEQ_512 = SeqScorerConfig(name="seqscorer_512x4096_d256_l2_h4", seed=42, input_dim=4096, d_model=256, n_heads=4,
                          n_layers=2, d_ff=768, max_steps=256, slots=512)


def _normal(shape, seed, tag, *ids):
    return keyed_rng(seed, tag, *ids).standard_normal(shape, dtype=np.float32)


def weights(cfg: SeqScorerConfig) -> dict:
    """fp32 arrays.  Linear maps are [out][in]."""
    s, D, d, f = cfg.seed, cfg.input_dim, cfg.d_model, cfg.d_ff
    lin = lambda o, i, *ids: _normal((o, i), s, *ids) / np.float32(np.sqrt(i))  # noqa: E731
    g = lambda n, *ids: (1 + 0.1 * _normal((n,), s, *ids)).astype(np.float32)  # noqa: E731
    b = lambda n, *ids: (0.1 * _normal((n,), s, *ids)).astype(np.float32)  # noqa: E731
    w = {"ln_in_g": g(D, TAG_LN_IN, 0), "ln_in_b": b(D, TAG_LN_IN, 1), "W_in": lin(d, D, TAG_WIN),
         "ln_out_g": g(d, TAG_OUT, 0), "ln_out_b": b(d, TAG_OUT, 1),
         "w_out": (_normal((d,), s, TAG_OUT, 2) / np.float32(np.sqrt(d))).astype(np.float32), "layers": []}
    for l in range(cfg.n_layers):
        w["layers"].append({
            "ln1_g": g(d, TAG_LAYER, l, 0), "ln1_b": b(d, TAG_LAYER, l, 1),
            "Wq": lin(d, d, TAG_LAYER, l, 2), "Wk": lin(d, d, TAG_LAYER, l, 3),
            "Wv": lin(d, d, TAG_LAYER, l, 4), "Wo": lin(d, d, TAG_LAYER, l, 5),
            "ln2_g": g(d, TAG_LAYER, l, 6), "ln2_b": b(d, TAG_LAYER, l, 7),
            "W1": lin(f, d, TAG_LAYER, l, 8), "W3": lin(f, d, TAG_LAYER, l, 9),
            "W2": lin(d, f, TAG_LAYER, l, 10)})
    return w


def step_states(cfg: SeqScorerConfig, rnd: int) -> np.ndarray:
    """bf16 bits [slots][D]: the step state each slot completes at round `rnd`."""
    return to_bf16_bits(_normal((cfg.slots, cfg.input_dim), cfg.seed, TAG_H, rnd))
