"""Seeded inputs and the event schedule of a tournament run (the full Alg. 1
loop: decode steps, thought boundaries, scheduler evictions, completions).

This module decides only what the outside world does - which prompt each
root trace starts from, the queries and new K/V of every step, the hidden
states at every thought boundary, when memory pressure makes the scheduler
evict, and which running trace finishes (answers are out of scope, so
completion is an event of the workload).  It performs none of the method's
arithmetic: no scores, ranking, eviction choice or block allocation.  Both
the oracle and the GPU run read it.

Every tensor is keyed: ``numpy.random.default_rng([seed, tag, *ids])`` with
tags 10 root prompt (root), 11 step queries (step), 12 step K/V (step),
13 thought-boundary hidden states (round), 14 probe weights, 15 completion
choice (step), 16 root prompt lengths.  Values are N(0, 1), rounded to bf16.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .generate import keyed_rng, to_bf16_bits

TAG_PROMPT, TAG_Q, TAG_KV, TAG_H, TAG_W, TAG_DONE, TAG_PLEN = 10, 11, 12, 13, 14, 15, 16


@dataclass(frozen=True)
class TournamentConfig:
    name: str
    seed: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    probe_dim: int
    slots: int           # trace slots of the pool (max_traces)
    capacity: int        # C
    swap_k: int          # K
    warmup: int          # w, in generated tokens
    interval: int        # a thought boundary (score update + tournament) every `interval` steps
    steps: int
    roots: int           # initial traces
    prompt_lo: int       # root prompt lengths ~ U[prompt_lo, prompt_hi]
    prompt_hi: int
    evict_every: int     # memory pressure: one eviction every `evict_every` steps (0: never)
    complete_every: int  # one running trace completes every `complete_every` steps (0: never)
    num_blocks: int
    max_blocks_per_trace: int


# A small run that exercises both cases, ghosts, warm-up and completions.
TOURNAMENT_SMALL = TournamentConfig(
    name="tournament_24slots_c16_k4", seed=21, n_q_heads=8, n_kv_heads=2, head_dim=128, probe_dim=256,
    slots=24, capacity=16, swap_k=4, warmup=6, interval=5, steps=80, roots=16, prompt_lo=5,
    prompt_hi=60, evict_every=9, complete_every=13, num_blocks=2048, max_blocks_per_trace=16)

# The paper's configuration (C = 256, K = 16; Sec. 5.1) at the Qwen3-8B layer
# shape, with warm-up and interval scaled to a few hundred decode steps.
TOURNAMENT_C256 = TournamentConfig(
    name="tournament_c256_k16_qwen3_8b", seed=22, n_q_heads=32, n_kv_heads=8, head_dim=128,
    probe_dim=4096, slots=320, capacity=256, swap_k=16, warmup=48, interval=16, steps=256, roots=256,
    prompt_lo=256, prompt_hi=1024, evict_every=40, complete_every=24, num_blocks=40000,
    max_blocks_per_trace=96)


class TournamentWorkload:
    def __init__(self, cfg: TournamentConfig):
        self.cfg = cfg

    def _normal(self, shape, tag, *ids):
        return keyed_rng(self.cfg.seed, tag, *ids).standard_normal(shape, dtype=np.float32)

    def prompt_lengths(self) -> list:
        c = self.cfg
        rng = keyed_rng(c.seed, TAG_PLEN)
        return [int(x) for x in rng.integers(c.prompt_lo, c.prompt_hi + 1, size=c.roots)]

    def prompt_kv(self, root: int, length: int):
        """bf16 bit patterns [length][Hkv][D] of K and V."""
        c = self.cfg
        x = self._normal((2, length, c.n_kv_heads, c.head_dim), TAG_PROMPT, root)
        return to_bf16_bits(x[0]), to_bf16_bits(x[1])

    def step_q(self, step: int, n: int) -> np.ndarray:
        """[n][Hq][D] bf16 bits for the step's n running traces, in list order."""
        c = self.cfg
        return to_bf16_bits(self._normal((n, c.n_q_heads, c.head_dim), TAG_Q, step))

    def step_kv(self, step: int, n: int):
        c = self.cfg
        x = self._normal((2, n, c.n_kv_heads, c.head_dim), TAG_KV, step)
        return to_bf16_bits(x[0]), to_bf16_bits(x[1])

    def round_h(self, rnd: int, n: int) -> np.ndarray:
        """[n][Dh] bf16 bits: the hidden states at the boundary, list order."""
        return to_bf16_bits(self._normal((n, self.cfg.probe_dim), TAG_H, rnd))

    def probe_weights(self):
        c = self.cfg
        w = self._normal((c.probe_dim,), TAG_W) / np.float32(np.sqrt(c.probe_dim))
        return w.astype(np.float32), 0.0

    def is_boundary(self, step: int) -> bool:
        return (step + 1) % self.cfg.interval == 0

    def evicts_at(self, step: int) -> bool:
        e = self.cfg.evict_every
        return e > 0 and (step + 1) % e == 0

    def completion_at(self, step: int, running: list):
        """The running trace (ascending id list) that completes at this step, or None."""
        c = self.cfg
        if c.complete_every <= 0 or (step + 1) % c.complete_every or len(running) < 2:
            return None
        k = int(keyed_rng(c.seed, TAG_DONE, step).integers(0, len(running)))
        return running[k]
