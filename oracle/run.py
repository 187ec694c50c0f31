"""Replay a synthetic workload through the oracle.  Test infrastructure only.

The schedule follows Alg. 1's main loop restricted to the hot path: every
step advances each live trace by one token (Generate) and attends over its
context; after every `interval` steps a round scores the traces at the
thought boundary, keeps the top `keep` and branches the top `n_parents`
into the freed slots (Tournament, Case 2 of Sec. 4.1 generalised to
`fanout` children per parent).
"""
from __future__ import annotations

import math

import numpy as np

from .attention import decode_attention
from .formats import bf16_to_f64
from .pool import PoolModel
from .probe import probe_scores, prune_branch_plan, rank


def sm_scale(head_dim: int) -> float:
    return 1.0 / math.sqrt(head_dim)


def new_pool(wl, num_blocks: int) -> PoolModel:
    c = wl.cfg
    return PoolModel(num_blocks=num_blocks, n_kv_heads=c.n_kv_heads, head_dim=c.head_dim,
                     kv_dtype=c.kv_dtype, max_traces=wl.T,
                     max_blocks_per_trace=c.max_blocks_per_trace, block_size=c.block_size)


def apply_setup(pool: PoolModel, wl, lazy: bool = True):
    """Run the workload's op log; node data is fetched lazily when `lazy`."""
    for op in wl.setup_ops():
        kind = op[0]
        if kind == "fork":
            pool.fork(op[1], op[2])
        elif kind == "alloc":
            pool.alloc(op[1], op[2])
        elif kind == "write":
            _, slot, pos0, nid = op
            n = wl.tree.nodes[nid].length
            if lazy and not wl.fp8:
                cache = {}

                def get(i, nid=nid, cache=cache):
                    if "kv" not in cache:
                        cache["kv"] = wl.node_kv(nid)
                    return cache["kv"][i]
                pool.write(slot, pos0, lambda g=get: g(0), lambda g=get: g(1), None, n=n)
            else:
                k, v, sc = wl.node_kv(nid)
                pool.write(slot, pos0, k, v, sc)
        else:
            raise ValueError(kind)


def attend(pool: PoolModel, wl, q_bits: np.ndarray, slots) -> dict:
    """Attention of the given slots; q_bits is the step's [T][Hq][D] bf16 array."""
    s = sm_scale(wl.cfg.head_dim)
    out = {}
    for t in slots:
        K, V = pool.materialise(t)
        out[t] = decode_attention(bf16_to_f64(q_bits[t]), K, V, s)
    return out


def run_round(pool: PoolModel, wl, rnd: int, ids, keep_override=None):
    """Probe, rank, prune, branch.  Returns (scores in list order, keep ids, pairs)."""
    c = wl.cfg
    h = wl.round_h(rnd)
    w, b = wl.probe_weights()
    ids = list(ids)
    scores = probe_scores(bf16_to_f64(h[ids]), w, b)
    keep = rank(ids, scores)[:c.keep] if keep_override is None else list(keep_override)
    freed, pairs = prune_branch_plan(ids, keep, c.n_parents)
    pool.free_traces(freed)
    if pairs:
        pool.fork([p for _, p in pairs], [ch for ch, _ in pairs])
    return scores, keep, pairs
