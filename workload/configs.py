"""Synthetic workload configurations for the population-decode hot path.

Each configuration describes one population of reasoning traces whose KV
caches share forked prefixes (a branch tree), the decode schedule that runs
over it, and the prune/branch rounds at thought boundaries.  The shapes are
the Qwen3-8B-style GQA layer (32 query heads, 8 KV heads, head dim 128) and
the Qwen3-32B-style layer (64/8/128) with fp8 E4M3 KV; the context lengths
follow the trace-length statistics the paper reports (median total trace
length in the tens of thousands of tokens, inherited prefixes of 14k-31k
tokens; Sec. 6 and App. A.5).

This module holds sizes only.  No part of the method's arithmetic lives here.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass


@dataclass(frozen=True)
class Config:
    name: str
    seed: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    kv_dtype: str            # "bf16" or "fp8_e4m3"
    probe_dim: int           # hidden size Dh of the probe input
    gens: tuple              # nodes per tree generation; gens[-1] == number of traces
    prompt_len: int          # shared root prompt above generation 1 (0: none)
    seg_lo: int              # segment lengths ~ U[seg_lo, seg_hi] (inclusive)
    seg_hi: int
    ctx_cap: int             # initial context + decode steps <= ctx_cap
    steps: int               # decode steps in the schedule
    interval: int            # prune/branch after every `interval` steps
    keep: int                # traces kept per round
    n_parents: int           # top kept traces that receive children
    block_size: int = 16

    @property
    def n_traces(self) -> int:
        return self.gens[-1]

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def fanout(self) -> int:
        return 1 + (self.n_traces - self.keep) // self.n_parents

    @property
    def kv_elem_bytes(self) -> int:
        return 1 if self.kv_dtype == "fp8_e4m3" else 2

    @property
    def max_blocks_per_trace(self) -> int:
        return -(-self.ctx_cap // self.block_size)

    def replace(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)


QWEN3_8B = dict(n_q_heads=32, n_kv_heads=8, head_dim=128)
QWEN3_32B = dict(n_q_heads=64, n_kv_heads=8, head_dim=128)

# 8 traces share one 512-token prefix and each own a 128-token suffix; one
# decode step, then a thought boundary: keep the top 4, fork each into 2.
CFG1 = Config(name="cfg1_8x641_qwen3_8b_bf16", seed=1, **QWEN3_8B, kv_dtype="bf16",
              probe_dim=4096, gens=(8,), prompt_len=512, seg_lo=128, seg_hi=128,
              ctx_cap=1024, steps=1, interval=1, keep=4, n_parents=4)

# 64 traces, 3-generation tree over a 1024-token prompt, segments U[512, 2048];
# 256 steps, round every 64 steps keeping 16, fork 4x.
CFG2 = Config(name="cfg2_64tr_3gen_qwen3_8b_bf16", seed=2, **QWEN3_8B, kv_dtype="bf16",
              probe_dim=4096, gens=(4, 16, 64), prompt_len=1024, seg_lo=512, seg_hi=2048,
              ctx_cap=8192, steps=256, interval=64, keep=16, n_parents=16)

# 256 traces, 4 generations, segments U[1k, 4k], contexts up to 16384;
# round every 128 steps keeping 64, fork 4x.
CFG3 = Config(name="cfg3_256tr_4gen_qwen3_8b_bf16", seed=3, **QWEN3_8B, kv_dtype="bf16",
              probe_dim=4096, gens=(4, 16, 64, 256), prompt_len=0, seg_lo=1024, seg_hi=4096,
              ctx_cap=16384, steps=512, interval=128, keep=64, n_parents=64)

# 512 traces, 5 generations, segments U[2k, 8k], contexts up to 32768;
# round every 256 steps keeping 128, fork 4x.  The HBM-bound steady state.
CFG4 = Config(name="cfg4_512tr_5gen_qwen3_8b_bf16", seed=4, **QWEN3_8B, kv_dtype="bf16",
              probe_dim=4096, gens=(2, 8, 32, 128, 512), prompt_len=0, seg_lo=2048,
              seg_hi=8192, ctx_cap=32768, steps=1024, interval=256, keep=128, n_parents=128)

# Qwen3-32B-style layer, 256 traces, 3 generations, contexts 4k-16k, fp8 E4M3 KV
# with one fp32 scale per (block, K|V); probe on 5120-d hidden states.
CFG5 = Config(name="cfg5_256tr_3gen_qwen3_32b_fp8", seed=5, **QWEN3_32B, kv_dtype="fp8_e4m3",
              probe_dim=5120, gens=(16, 64, 256), prompt_len=0, seg_lo=1366, seg_hi=5461,
              ctx_cap=16896, steps=512, interval=128, keep=64, n_parents=64)

CONFIGS = {1: CFG1, 2: CFG2, 3: CFG3, 4: CFG4, 5: CFG5}


def tiny(kv_dtype: str = "bf16", **kw) -> Config:
    """A small configuration the oracle finishes in well under a second.

    Several tiles per unit and ragged (non-block-aligned) segments, so forks
    create tail copies.
    """
    base = dict(name="tiny", seed=11, n_q_heads=8, n_kv_heads=2, head_dim=128,
                kv_dtype=kv_dtype, probe_dim=256, gens=(2, 4, 8), prompt_len=37,
                seg_lo=9, seg_hi=70, ctx_cap=512, steps=40, interval=16, keep=4,
                n_parents=2)
    base.update(kw)
    return Config(**base)
