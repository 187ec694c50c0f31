"""Drive a synthetic population workload through libgambit on one GPU.

Setup replays the workload's op log (alloc / write / fork) into a pool; a
decode step appends one token per trace and attends; after every
`interval` steps a round scores, ranks, prunes and branches (Alg. 1
Generate and Tournament, restricted to the attention, probe and
prune/branch work).
"""
from __future__ import annotations

import time

import numpy as np
import torch

from .gambit import Pool

BS = 16


def _to_dev(a, dtype: torch.dtype, device) -> torch.Tensor:
    if isinstance(a, torch.Tensor):  # already resident (e.g. kept from an earlier replay)
        return a
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype == torch.bfloat16:
        t = t.view(torch.int16).view(torch.bfloat16)
    return t.to(device, non_blocking=False)


def estimate_blocks(wl, total_steps: int | None = None) -> int:
    """Blocks the schedule can ever hold at once, with margin."""
    c, tr = wl.cfg, wl.tree
    steps = wl.total_steps if total_steps is None else total_steps
    blocks = 0
    for n in tr.nodes:
        first = n.start // BS
        last = (n.start + n.length - 1) // BS
        blocks += last - first + 1 + 1          # blocks it spans + a tail copy per fork
    blocks += c.n_traces * (steps // BS + 2)      # decode growth
    n_rounds = steps // c.interval + 1
    blocks += n_rounds * (c.n_traces - c.keep) * (steps // BS + 2)  # children's private growth
    return int(blocks * 1.05) + 64


class PopulationRun:
    def __init__(self, wl, *, device: str = "cuda", num_blocks: int | None = None,
                 max_splits: int = 0, verbose: bool = False):
        self.wl, self.cfg = wl, wl.cfg
        self.device = device
        self.T = wl.T
        self.ids = np.arange(self.T, dtype=np.int32)
        self.fp8 = wl.fp8
        self.cache_dtype = torch.uint8 if self.fp8 else torch.bfloat16
        nb = num_blocks or estimate_blocks(wl)
        self.pool = Pool(num_blocks=nb, num_q_heads=self.cfg.n_q_heads,
                         num_kv_heads=self.cfg.n_kv_heads, max_traces=self.T,
                         max_blocks_per_trace=self.cfg.max_blocks_per_trace,
                         kv_dtype=self.cfg.kv_dtype, max_splits=max_splits, device=device)
        self.verbose = verbose
        self.q = {}
        self.kv = {}
        w, b = wl.probe_weights()
        self.w = torch.from_numpy(w).to(device)
        self.b = b
        self.h = {}

    def log(self, msg):
        if self.verbose:
            print(f"[runner] {msg}", flush=True)

    # ------------------------------------------------------------ setup --
    def setup(self, node_data=None):
        """Replay the op log.  node_data(nid) -> (k, v, scales) defaults to the generator."""
        get = node_data or self.wl.node_kv
        t0 = time.time()
        for op in self.wl.setup_ops():
            if op[0] == "fork":
                self.pool.kv_fork(op[1], op[2])
            elif op[0] == "alloc":
                self.pool.kv_alloc(op[1], op[2])
            else:
                _, slot, pos0, nid = op
                k, v, sc = get(nid)
                kd = _to_dev(k, self.cache_dtype, self.device)
                vd = _to_dev(v, self.cache_dtype, self.device)
                self.pool.kv_write(slot, pos0, kd, vd, sc)
        torch.cuda.synchronize()
        self.log(f"setup done in {time.time() - t0:.1f}s")

    # ------------------------------------------------------------ inputs --
    def load_steps(self, steps, keep_host: bool = False):
        """Generate and upload the queries and new K/V of the given steps.

        With keep_host the host arrays stay in self.host[s] = (q, k, v)."""
        steps = [s for s in steps if s not in self.q]
        wl = self.wl
        if keep_host and not hasattr(self, "host"):
            self.host = {}

        def gen(s):
            return s, wl.step_q(s), wl.step_kv(s)
        for i in range(0, len(steps), 64):
            for s, q, (k, v) in wl.many(gen, steps[i:i + 64]):
                self.q[s] = _to_dev(q, torch.bfloat16, self.device)
                self.kv[s] = (_to_dev(k, self.cache_dtype, self.device),
                              _to_dev(v, self.cache_dtype, self.device))
                if keep_host:
                    self.host[s] = (q, k, v)

    def share_inputs(self, other: "PopulationRun"):
        """Use another run's resident step and round inputs (same workload)."""
        self.q, self.kv, self.h = other.q, other.kv, other.h

    def load_rounds(self, rounds):
        for r in rounds:
            if r not in self.h:
                self.h[r] = _to_dev(self.wl.round_h(r), torch.bfloat16, self.device)

    # ------------------------------------------------------------ steps --
    def decode(self, s: int, out: torch.Tensor | None = None, out_dtype=torch.bfloat16):
        k, v = self.kv[s]
        return self.pool.decode_attn(self.ids, self.q[s], k, v, out=out, out_dtype=out_dtype)

    def round(self, r: int):
        c = self.cfg
        return self.pool.score_prune_branch(self.ids, self.h[r], self.w, self.b, c.keep, c.n_parents)

    def schedule(self):
        """[(step, round or None)] of the workload."""
        after = {s: i for i, s in enumerate(self.wl.rounds_after())}
        return [(s, after.get(s)) for s in range(self.wl.total_steps)]
