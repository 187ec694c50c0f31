"""Seeded synthetic inputs for the population-decode hot path.

This module is the ONLY code that both the oracle and the GPU path use.  It
draws random numbers, rounds them to the storage formats (bf16 round-to-
nearest-even, OCP E4M3FN with saturation), lays out the branch tree and emits
the operation log that builds it.  It performs none of the method's
arithmetic: no attention, no probe, no ranking, no block allocation.

Every tensor is keyed, so any piece can be regenerated on its own:
``numpy.random.default_rng([cfg.seed, tag, *ids])`` with tags

  0  segment K/V of tree node ``node`` (chunked by 256 tokens)
  1  per-step queries            (step)
  2  per-step new K/V            (step)
  3  per-round probe inputs h    (round)
  4  probe weights w
  5  segment lengths             (generation, node index)

Values are N(0, 1) drawn in float32.  Tree shape: generation g has
gens[g] nodes and node i of generation g+1 hangs under node i // F of
generation g (F = gens[g+1] // gens[g]), so every node at one level has F
children.  An optional shared prompt sits above generation 1.  Leaves map to
trace slots 0..T-1 in order; an internal node is owned by the slot of its
leftmost leaf.  The op log writes each node into its owner slot, then forks
that slot into the owner slots of the node's other children (Branch: a child
starts from its parent's prefix by sharing its KV, Alg. 1 notation and
Sec. 4.1 Case 2).
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

from .configs import Config

TAG_SEG, TAG_Q, TAG_KVNEW, TAG_H, TAG_W, TAG_LEN = 0, 1, 2, 3, 4, 5
SEG_CHUNK = 256                      # tokens per independently keyed KV chunk
FP8_MAX = 448.0                      # largest finite OCP E4M3FN magnitude
FP8_MIN_SCALE = 2.0 ** -20
FP8_APPEND_SCALE = 2.0 ** -6         # scale of blocks a decode step allocates

_THREADS = max(1, min(16, len(os.sched_getaffinity(0))))


def keyed_rng(seed: int, tag: int, *ids: int) -> np.random.Generator:
    return np.random.default_rng([int(seed), int(tag), *[int(i) for i in ids]])


# ---------------------------------------------------------------- formats ---
def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest even."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def to_e4m3_bytes(x: np.ndarray, scale) -> np.ndarray:
    """x / scale -> OCP E4M3FN codes (uint8), saturating at +-448, RNE."""
    import torch
    y = np.clip(np.asarray(x, np.float32) / np.asarray(scale, np.float32), -FP8_MAX, FP8_MAX)
    t = torch.from_numpy(np.ascontiguousarray(y, dtype=np.float32))
    return t.to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def e4m3_block_scale(amax: float) -> float:
    return float(np.float32(max(amax / FP8_MAX, FP8_MIN_SCALE)))


# ------------------------------------------------------------------ tree ---
@dataclass
class Node:
    nid: int
    gen: int                  # 0 = shared prompt, 1.. = generations
    parent: int               # node id, -1 for a root
    length: int               # tokens in this segment
    start: int                # position of its first token in every trace below it
    slot: int                 # owner slot (leftmost leaf)
    children: list = field(default_factory=list)


@dataclass
class Tree:
    cfg: Config
    total_steps: int
    nodes: list
    leaves: list              # node id of the leaf of slot t
    init_len: np.ndarray      # [T] initial context length per slot

    def path(self, slot: int) -> list:
        out, n = [], self.leaves[slot]
        while n >= 0:
            out.append(n)
            n = self.nodes[n].parent
        return out[::-1]


def build_tree(cfg: Config, total_steps: int | None = None) -> Tree:
    """Lay out the branch tree; truncate segments so context + steps <= cap."""
    steps = cfg.steps if total_steps is None else int(total_steps)
    budget = cfg.ctx_cap - steps
    levels = list(cfg.gens)
    depth = len(levels)
    if budget < depth + (1 if cfg.prompt_len else 0):
        raise ValueError("context cap too small for the schedule")
    nodes: list[Node] = []
    T = levels[-1]
    prev = []
    if cfg.prompt_len:
        plen = min(cfg.prompt_len, budget - depth)
        nodes.append(Node(0, 0, -1, plen, 0, 0))
        prev = [0]
    for g, cnt in enumerate(levels, start=1):
        cur = []
        lens = keyed_rng(cfg.seed, TAG_LEN, g).integers(cfg.seg_lo, cfg.seg_hi + 1, size=cnt)
        fan = cnt // len(prev) if prev else 0
        if prev and cnt % len(prev):
            raise ValueError("generation sizes must divide")
        for i in range(cnt):
            par = prev[i // fan] if prev else -1
            start = nodes[par].start + nodes[par].length if par >= 0 else 0
            below = depth - g                    # levels still to come under this node
            ln = int(min(lens[i], budget - start - below))
            ln = max(ln, 1)
            nid = len(nodes)
            nodes.append(Node(nid, g, par, ln, start, -1))
            if par >= 0:
                nodes[par].children.append(nid)
            cur.append(nid)
        prev = cur
    leaves = prev
    assert len(leaves) == T
    for t, nid in enumerate(leaves):
        n = nid
        while n >= 0 and nodes[n].slot < 0:
            nodes[n].slot = t
            n = nodes[n].parent
    if cfg.prompt_len:
        nodes[0].slot = 0
    init_len = np.array([nodes[n].start + nodes[n].length for n in leaves], np.int64)
    assert init_len.max() + steps <= cfg.ctx_cap
    return Tree(cfg, steps, nodes, leaves, init_len)


def setup_ops(tree: Tree) -> list:
    """Operation log that builds the initial population, generation by generation.

    ("fork", parents, children) - child slots start from the parent's prefix
    ("alloc", slots, n_tokens)  - extend each slot by n tokens
    ("write", slot, pos0, nid)  - write node nid's K/V at positions pos0...
    """
    ops = []
    by_gen: dict[int, list] = {}
    for n in tree.nodes:
        by_gen.setdefault(n.gen, []).append(n)
    for g in sorted(by_gen):
        gen_nodes = by_gen[g]
        pairs = [(tree.nodes[n.parent].slot, n.slot) for n in gen_nodes
                 if n.parent >= 0 and n.slot != tree.nodes[n.parent].slot]
        if pairs:
            ops.append(("fork", [p for p, _ in pairs], [c for _, c in pairs]))
        ops.append(("alloc", [n.slot for n in gen_nodes], [n.length for n in gen_nodes]))
        for n in gen_nodes:
            ops.append(("write", n.slot, n.start, n.nid))
    return ops


# ------------------------------------------------------------- generator ---
class Workload:
    """All inputs of one configuration, generated on demand from keys."""

    def __init__(self, cfg: Config, total_steps: int | None = None):
        self.cfg = cfg
        self.tree = build_tree(cfg, total_steps)
        self.total_steps = self.tree.total_steps
        self.T = cfg.n_traces
        self.fp8 = cfg.kv_dtype == "fp8_e4m3"
        if self.fp8 and cfg.interval < cfg.block_size and self.total_steps > cfg.interval:
            raise ValueError("fp8 workloads need interval >= block size")
        self._tail_scale: dict[int, np.ndarray] = {}

    # -- schedule
    def rounds_after(self) -> list:
        """Steps s after which a prune/branch round runs (0-based)."""
        P = self.cfg.interval
        return [s for s in range(self.total_steps) if (s + 1) % P == 0]

    def setup_ops(self) -> list:
        return setup_ops(self.tree)

    # -- raw float data
    def node_f32(self, nid: int) -> np.ndarray:
        """[2][len][Hkv][D] float32 (K, V) of a tree node."""
        c = self.cfg
        n = self.tree.nodes[nid].length
        out = np.empty((2, n, c.n_kv_heads, c.head_dim), np.float32)
        chunks = range(0, n, SEG_CHUNK)

        def fill(c0):
            cnt = min(SEG_CHUNK, n - c0)
            out[:, c0:c0 + cnt] = keyed_rng(c.seed, TAG_SEG, nid, c0 // SEG_CHUNK).standard_normal(
                (2, cnt, c.n_kv_heads, c.head_dim), dtype=np.float32)
        if n > 4 * SEG_CHUNK and _THREADS > 1:
            with ThreadPoolExecutor(_THREADS) as ex:
                list(ex.map(fill, chunks))
        else:
            for c0 in chunks:
                fill(c0)
        return out

    # -- stored K/V of a node
    def node_kv(self, nid: int):
        """Returns (k, v, scales).

        bf16: k, v are uint16 bit patterns [len][Hkv][D]; scales is None.
        fp8:  k, v are E4M3FN codes [len][Hkv][D]; scales is float32
              [n_started][2] (K, V) for the blocks whose first position lies
              inside this node, in ascending order.  Tokens that land in a block
              started by an ancestor are quantised with that block's scale.
        """
        x = self.node_f32(nid)
        if not self.fp8:
            b = to_bf16_bits(x)
            return b[0], b[1], None
        node = self.tree.nodes[nid]
        BS = self.cfg.block_size
        n, s0 = node.length, node.start
        per_tok = np.ones((n, 2), np.float32)
        started = []
        pos = s0
        while pos < s0 + n:
            blk = pos // BS
            hi = min((blk + 1) * BS, s0 + n)
            lo_i, hi_i = pos - s0, hi - s0
            if pos % BS == 0:
                sc = np.array([e4m3_block_scale(float(np.abs(x[0, lo_i:hi_i]).max())),
                               e4m3_block_scale(float(np.abs(x[1, lo_i:hi_i]).max()))], np.float32)
                started.append(sc)
            else:
                sc = self._inherited_tail_scale(node)
            per_tok[lo_i:hi_i] = sc
            pos = hi
        self._tail_scale[nid] = per_tok[-1].copy()
        k = to_e4m3_bytes(x[0], per_tok[:, 0, None, None])
        v = to_e4m3_bytes(x[1], per_tok[:, 1, None, None])
        scales = np.array(started, np.float32).reshape(-1, 2)
        return k, v, scales

    def _inherited_tail_scale(self, node: Node) -> np.ndarray:
        if node.parent < 0:
            raise AssertionError("a root starts at position 0")
        if node.parent not in self._tail_scale:
            self.node_kv(node.parent)
        return self._tail_scale[node.parent]

    def tail_scale_of_slot(self, slot: int) -> np.ndarray:
        leaf = self.tree.leaves[slot]
        if leaf not in self._tail_scale:
            self.node_kv(leaf)
        return self._tail_scale[leaf]

    # -- per-step inputs (slot-indexed, independent of which traces are live)
    def step_q(self, step: int) -> np.ndarray:
        c = self.cfg
        x = keyed_rng(c.seed, TAG_Q, step).standard_normal(
            (self.T, c.n_q_heads, c.head_dim), dtype=np.float32)
        return to_bf16_bits(x)

    def step_kv_f32(self, step: int) -> np.ndarray:
        c = self.cfg
        return keyed_rng(c.seed, TAG_KVNEW, step).standard_normal(
            (2, self.T, c.n_kv_heads, c.head_dim), dtype=np.float32)

    def step_kv(self, step: int):
        """New K/V of every slot at `step`: [T][Hkv][D] each (bf16 bits or E4M3 codes).

        For fp8, a token that lands in a slot's initial, partly filled tail
        block is quantised with that block's scale; every later token lands in
        a block allocated by a decode step (scale 2^-6), because a round runs
        only after at least one block's worth of steps.
        """
        x = self.step_kv_f32(step)
        if not self.fp8:
            b = to_bf16_bits(x)
            return b[0], b[1]
        BS = self.cfg.block_size
        sc = np.full((self.T, 2), FP8_APPEND_SCALE, np.float32)
        for t in range(self.T):
            L0 = int(self.tree.init_len[t])
            if L0 % BS and step < BS - L0 % BS and step < self.cfg.interval:
                sc[t] = self.tail_scale_of_slot(t)
        k = to_e4m3_bytes(x[0], sc[:, 0, None, None])
        v = to_e4m3_bytes(x[1], sc[:, 1, None, None])
        return k, v

    def round_h(self, rnd: int) -> np.ndarray:
        c = self.cfg
        x = keyed_rng(c.seed, TAG_H, rnd).standard_normal((self.T, c.probe_dim), dtype=np.float32)
        return to_bf16_bits(x)

    def probe_weights(self):
        c = self.cfg
        w = keyed_rng(c.seed, TAG_W).standard_normal(c.probe_dim) / math.sqrt(c.probe_dim)
        return w.astype(np.float32), 0.0

    # -- bulk helpers (threaded)
    def many(self, fn, keys):
        if _THREADS > 1 and len(keys) > 1:
            with ThreadPoolExecutor(_THREADS) as ex:
                return list(ex.map(fn, keys))
        return [fn(k) for k in keys]
