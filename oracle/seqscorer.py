"""The history-aware sequence scorer of App. A.1 (Eqs. 4-6).  Test
infrastructure only.

For one trace with step states h_1 .. h_T (the hidden state at each thought
boundary), in fp64:

    x_t   = GELU(W_in LN(h_t))                                  (Eq. 4)
    z_1..z_T = Transformer(x_1..x_T)                            (Eq. 5)
    y_t   = sigmoid(w_out . LN(z_t))                            (Eq. 6)

Each Transformer layer is a pre-norm residual block pair (the paper names
the parts, not their order): x += Wo MHA(LN1(x)), causal, with RoPE on
queries and keys at the step index (0-based), then x += W2 (SiLU(W1 LN2(x))
* W3 LN2(x)) (SwiGLU).  LN is LayerNorm with gain and bias, eps 1e-5; GELU is
the erf form; attention scale 1/sqrt(head_dim); RoPE rotates the two halves
of each head (x_i, x_{i+hd/2}) by angle pos * 10000^(-2i/hd); no biases in
the linear maps (Eqs. 4 and 6 have none).  The scorer's value for a trace
at a boundary is y_T at its last step (Eq. 7 trains only that position);
position t depends on steps 1..t only.

The oracle computes the whole sequence each time (no cache); the GPU path
computes one new step per boundary against cached keys and values.
"""
from __future__ import annotations

import math

import numpy as np

LN_EPS = 1e-5
ROPE_BASE = 10000.0


def layer_norm(x: np.ndarray, g, b) -> np.ndarray:
    x = np.asarray(x, np.float64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + LN_EPS) * np.asarray(g, np.float64) + np.asarray(b, np.float64)


def gelu(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x, np.float64)
    erf = np.vectorize(math.erf)
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def silu(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x, np.float64)
    return x / (1.0 + np.exp(-x))


def rope(x: np.ndarray, pos: np.ndarray) -> np.ndarray:
    """x [T][hd], pos [T]: each pair (x_i, x_{i+hd/2}) rotated by pos * base^(-2i/hd)."""
    hd = x.shape[-1]
    half = hd // 2
    theta = ROPE_BASE ** (-np.arange(half, dtype=np.float64) * 2.0 / hd)
    ang = np.asarray(pos, np.float64)[:, None] * theta[None, :]
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[:, :half], x[:, half:]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=1)


def causal_mha(x: np.ndarray, Wq, Wk, Wv, Wo, n_heads: int) -> np.ndarray:
    """x [T][d] -> Wo . concat_heads(softmax(q k^T / sqrt(hd), causal) v)."""
    T, d = x.shape
    hd = d // n_heads
    q = x @ np.asarray(Wq, np.float64).T
    k = x @ np.asarray(Wk, np.float64).T
    v = x @ np.asarray(Wv, np.float64).T
    pos = np.arange(T)
    out = np.empty((T, d))
    for h in range(n_heads):
        sl = slice(h * hd, (h + 1) * hd)
        qh, kh = rope(q[:, sl], pos), rope(k[:, sl], pos)
        s = qh @ kh.T / math.sqrt(hd)
        s = np.where(np.tril(np.ones((T, T), bool)), s, -np.inf)
        p = np.exp(s - s.max(axis=1, keepdims=True))
        p /= p.sum(axis=1, keepdims=True)
        out[:, sl] = p @ v[:, sl]
    return out @ np.asarray(Wo, np.float64).T


def swiglu(x: np.ndarray, W1, W3, W2) -> np.ndarray:
    a = x @ np.asarray(W1, np.float64).T
    b = x @ np.asarray(W3, np.float64).T
    return (silu(a) * b) @ np.asarray(W2, np.float64).T


def scorer_outputs(w: dict, H: np.ndarray, n_heads: int) -> np.ndarray:
    """H [T][D] step states (fp64 values) -> y [T], y_t conditioned on steps 1..t."""
    H = np.asarray(H, np.float64)
    x = gelu(layer_norm(H, w["ln_in_g"], w["ln_in_b"]) @ np.asarray(w["W_in"], np.float64).T)
    for L in w["layers"]:
        x = x + causal_mha(layer_norm(x, L["ln1_g"], L["ln1_b"]), L["Wq"], L["Wk"], L["Wv"], L["Wo"], n_heads)
        x = x + swiglu(layer_norm(x, L["ln2_g"], L["ln2_b"]), L["W1"], L["W3"], L["W2"])
    logit = layer_norm(x, w["ln_out_g"], w["ln_out_b"]) @ np.asarray(w["w_out"], np.float64)
    return 1.0 / (1.0 + np.exp(-logit))


class SeqScorerModel:
    """Per-slot step histories: a boundary appends each listed trace's step
    state and scores it; a fork gives the child the parent's history (the
    child's trace is the parent's prefix); a freed slot forgets its history."""

    def __init__(self, w: dict, n_heads: int, slots: int, max_steps: int):
        self.w, self.n_heads, self.max_steps = w, n_heads, max_steps
        self.hist = [[] for _ in range(slots)]

    def step(self, ids, H) -> np.ndarray:
        out = []
        for i, t in enumerate(ids):
            if len(self.hist[t]) >= self.max_steps:
                raise ValueError(f"trace {t} holds {self.max_steps} steps")
            self.hist[t].append(np.asarray(H[i], np.float64))
            out.append(scorer_outputs(self.w, np.stack(self.hist[t]), self.n_heads)[-1])
        return np.array(out)

    def fork(self, parents, children):
        for p, c in zip(parents, children):
            self.hist[c] = list(self.hist[p])

    def free(self, ids):
        for t in ids:
            self.hist[t] = []
