"""Decode-step attention by definition, fp64.  Test infrastructure only.

For one trace with context K, V in R^{L x Hkv x D} (every token it
inherited through forks plus every token it appended itself, including the
current step's token) and query q in R^{Hq x D}, query head h reads KV head
h // (Hq / Hkv) and

    s_j = scale * <q_h, K[j, h // g]>
    p_j = exp(s_j - max_k s_k) / sum_k exp(s_k - max_k s_k)
    o_h = sum_j p_j V[j, h // g]

The softmax scale is passed in (1/sqrt(D) for the workloads).  A forked
child and a trace holding a private copy of the same prefix have the same K,
V rows, so the result depends only on the token sequence, never on how the
pool stores it (Alg. 1 notation, Branch; Sec. 4.1 Case 2).
"""
from __future__ import annotations

import numpy as np


def softmax_weights(q: np.ndarray, K: np.ndarray, scale: float) -> np.ndarray:
    """p[h, j] for every query head h and context position j."""
    q = np.asarray(q, np.float64)
    K = np.asarray(K, np.float64)
    Hq, Hkv = q.shape[0], K.shape[1]
    g = Hq // Hkv
    p = np.empty((Hq, K.shape[0]), np.float64)
    for h in range(Hq):
        s = (K[:, h // g, :] @ q[h]) * scale
        e = np.exp(s - s.max())
        p[h] = e / e.sum()
    return p


def decode_attention(q: np.ndarray, K: np.ndarray, V: np.ndarray, scale: float) -> np.ndarray:
    """o[h, :] for one trace.  q: [Hq][D]; K, V: [L][Hkv][D]; returns [Hq][D] fp64."""
    if K.shape[0] == 0:
        raise ValueError("a trace attends over at least its current token")
    V = np.asarray(V, np.float64)
    Hq, Hkv = q.shape[0], K.shape[1]
    g = Hq // Hkv
    p = softmax_weights(q, K, scale)
    out = np.empty((Hq, V.shape[2]), np.float64)
    for h in range(Hq):
        out[h] = p[h] @ V[:, h // g, :]
    return out
