"""Probe scores, ranking and the prune/branch plan.  Test infrastructure only.

* Probe: z_t = sum_i h_{t,i} w_i + b and score_t = 1 / (1 + e^{-z_t}), the
  sigmoid head sigma(w^T x) of Eq. 6 applied directly to the boundary hidden
  state h (the light-weight scorer f_theta of Sec. 4.1).
* Ranking: traces ordered by score, highest first (Alg. 1 Tournament, and
  the ordered list tau_(1) >= ... >= tau_(n) of Sec. 4.1); equal scores go
  to the lower trace id.
* Prune/branch (Eq. 3, generalised): the traces outside the top `keep` are
  freed in ascending id order; the freed slots, ascending, receive the
  children; with c = (n - keep) / n_parents children per parent, child j
  descends from the kept trace of rank j // c.  The parent keeps running
  (App. A.5: a branching event is a split in which the parent continues).
  The paper's Case 2 is keep = C - K, n_parents = K (c = 1).
"""
from __future__ import annotations

import math

import numpy as np


def probe_logits(h: np.ndarray, w: np.ndarray, b: float) -> np.ndarray:
    return np.asarray(h, np.float64) @ np.asarray(w, np.float64) + float(b)


def sigmoid(z: np.ndarray) -> np.ndarray:
    z = np.asarray(z, np.float64)
    return np.array([1.0 / (1.0 + math.exp(-float(x))) if x > -700 else 0.0 for x in z.ravel()],
                    np.float64).reshape(z.shape)


def probe_scores(h: np.ndarray, w: np.ndarray, b: float) -> np.ndarray:
    return sigmoid(probe_logits(h, w, b))


def rank(trace_ids, scores) -> list:
    """Trace ids ordered by (score descending, trace id ascending)."""
    ids = [int(t) for t in trace_ids]
    sc = [float(s) for s in scores]
    order = sorted(range(len(ids)), key=lambda i: (-sc[i], ids[i]))
    return [ids[i] for i in order]


def prune_branch_plan(trace_ids, keep_ids, n_parents: int):
    """(freed ids ascending, [(child, parent)] in child order)."""
    ids = [int(t) for t in trace_ids]
    keep = [int(t) for t in keep_ids]
    n, k = len(ids), len(keep)
    if not (0 < n_parents <= k <= n) or (n - k) % n_parents:
        raise ValueError("keep / n_parents do not divide the population")
    kept = set(keep)
    freed = sorted(t for t in ids if t not in kept)
    c = (n - k) // n_parents
    pairs = [(child, keep[j // c]) for j, child in enumerate(freed)] if c else []
    return freed, pairs
