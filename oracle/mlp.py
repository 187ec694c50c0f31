"""The 2-layer MLP scorer on a thought-boundary hidden state.  Test
infrastructure only.

The paper's main evaluation scores traces with STEP's ready-made two-layer
MLP on the last-layer hidden state h at a thought boundary (Sec. 4.1
and Sec. 5.1: f_theta takes h_{i,j} and returns a score in [0, 1]); it gives
no dimensions, activation or weights.  This module states the plain form:

    f(h) = sigmoid( w2 . act(W1 h + b1) + b2 ),   act = ReLU or GELU (erf),

computed in fp64 over the bf16-decoded h and W1 and the fp32 b1, w2, b2.
"""
from __future__ import annotations

import math

import numpy as np

ACTS = ("relu", "gelu")


def activation(x: np.ndarray, act: str) -> np.ndarray:
    x = np.asarray(x, np.float64)
    if act == "relu":
        return np.maximum(x, 0.0)
    if act == "gelu":  # x * Phi(x), Phi the standard normal CDF
        return np.array([v * 0.5 * (1.0 + math.erf(v / math.sqrt(2.0))) for v in x.ravel()]).reshape(x.shape)
    raise ValueError(act)


def mlp_logits(h: np.ndarray, W1: np.ndarray, b1: np.ndarray, w2: np.ndarray, b2: float, act: str) -> np.ndarray:
    """h [n][Dh], W1 [H1][Dh], b1 [H1], w2 [H1]  ->  logits [n]."""
    z = np.asarray(h, np.float64) @ np.asarray(W1, np.float64).T + np.asarray(b1, np.float64)
    return activation(z, act) @ np.asarray(w2, np.float64) + float(b2)


def mlp_scores(h, W1, b1, w2, b2, act) -> np.ndarray:
    z = mlp_logits(h, W1, b1, w2, b2, act)
    return np.array([1.0 / (1.0 + math.exp(-float(v))) if v > -700 else 0.0 for v in z], np.float64)
