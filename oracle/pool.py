"""Model of the refcounted paged KV pool.  Test infrastructure only.

Two things are modelled, independently of each other:

1. The token sequence of every trace (what attention reads).  A trace's
   content is a list of runs over its positions; fork gives the child its
   own copy of the parent's list (the per-trace copy the method avoids on
   the GPU; Sec. 4.1 Case 2: the child reuses its parent's KV).
2. The physical block bookkeeping (what the block tables must say):

   * allocation takes the lowest free block id; requests are served in the
     call's list order and, within a trace, in ascending logical index;
   * fork: the child row lists the parent's full blocks (each refcount + 1);
     a partial last block is copied into one newly allocated block; the
     child's length equals the parent's (Alg. 1 notation: Branch starts the
     child from its parent's prefix, whose KV it shares);
   * free: every referenced block loses one reference and becomes free at
     zero; the row empties and the length drops to 0 (Sec. 4.1 Case 2:
     pruning frees the non-shared blocks);
   * a decode step appends one token per listed trace, taking a new block
     when the length is a multiple of the block size.

fp8 pools keep one (K, V) scale per block: a block allocated by an explicit
allocation starts at (1, 1), one allocated by a decode step at the pool's
append scale, a write sets the scales of the blocks whose first position it
covers, and the copied tail block carries its scales.  A stored value is the
decoded code times its block's scale.
"""
from __future__ import annotations

import heapq

import numpy as np

from .formats import bf16_to_f64, decode, quantise_e4m3fn


class PoolError(ValueError):
    def __init__(self, code: str, msg: str = ""):
        super().__init__(f"{code}: {msg}")
        self.code = code


def _resolve(src):
    return src() if callable(src) else src


class PoolModel:
    def __init__(self, *, num_blocks: int, n_kv_heads: int, head_dim: int, kv_dtype: str,
                 max_traces: int, max_blocks_per_trace: int, block_size: int = 16,
                 append_scale: float = 2.0 ** -6):
        self.BS = block_size
        self.Hkv, self.D = n_kv_heads, head_dim
        self.kv_dtype = kv_dtype
        self.fp8 = kv_dtype == "fp8_e4m3"
        self.num_blocks = num_blocks
        self.max_traces = max_traces
        self.max_blocks = max_blocks_per_trace
        self.append_scale = float(np.float32(append_scale))
        self.free = list(range(num_blocks))
        heapq.heapify(self.free)
        self.refcount = [0] * num_blocks
        self.table = [[] for _ in range(max_traces)]
        self.seq_len = [0] * max_traces
        # runs[t]: list of [pos_lo, pos_hi, ksrc, vsrc, src_lo]; ksrc/vsrc are
        # code arrays [n][Hkv][D] (or callables returning them)
        self.runs = [[] for _ in range(max_traces)]
        self.bscale = [[] for _ in range(max_traces)]

    # ------------------------------------------------------------ helpers --
    def _nblocks(self, L: int) -> int:
        return -(-L // self.BS)

    def _check_ids(self, ids, what="trace"):
        seen = set()
        for t in ids:
            if not (0 <= t < self.max_traces):
                raise PoolError("INVALID", f"{what} id {t} out of range")
            if t in seen:
                raise PoolError("INVALID", f"duplicate {what} id {t}")
            seen.add(t)

    def _take_block(self) -> int:
        return heapq.heappop(self.free)

    def used_blocks(self) -> int:
        return self.num_blocks - len(self.free)

    # -------------------------------------------------------------- alloc --
    def alloc(self, ids, n_tokens):
        ids = [int(t) for t in ids]
        n_tokens = [int(n) for n in n_tokens]
        self._check_ids(ids)
        need = 0
        for t, n in zip(ids, n_tokens):
            if n < 0:
                raise PoolError("INVALID", "negative token count")
            L = self.seq_len[t]
            if self._nblocks(L + n) > self.max_blocks:
                raise PoolError("INVALID", "trace exceeds max_blocks_per_trace")
            need += self._nblocks(L + n) - self._nblocks(L)
        if need > len(self.free):
            raise PoolError("OUT_OF_BLOCKS", f"need {need}, free {len(self.free)}")
        for t, n in zip(ids, n_tokens):
            self._grow(t, n, (1.0, 1.0))

    def _grow(self, t: int, n: int, scale):
        L = self.seq_len[t]
        for _ in range(self._nblocks(L + n) - self._nblocks(L)):
            b = self._take_block()
            self.refcount[b] = 1
            self.table[t].append(b)
            self.bscale[t].append(tuple(scale))
        self.seq_len[t] = L + n

    # -------------------------------------------------------------- write --
    def write(self, t: int, pos0: int, k, v, scales=None, n: int | None = None):
        """k, v: codes [n][Hkv][D] (or callables returning them, with n given)."""
        if n is None:
            n = int(np.asarray(k).shape[0])
        if not (0 <= t < self.max_traces):
            raise PoolError("INVALID", "trace id out of range")
        if pos0 < 0 or n < 0 or pos0 + n > self.seq_len[t]:
            raise PoolError("INVALID", "write outside the allocated positions")
        if n == 0:
            return
        BS = self.BS
        for j in range(pos0 // BS, (pos0 + n - 1) // BS + 1):
            if self.refcount[self.table[t][j]] != 1:
                raise PoolError("SHARED_WRITE", f"block {j} of trace {t} is shared")
        started = [j for j in range((pos0 + BS - 1) // BS, (pos0 + n - 1) // BS + 1)
                   if j * BS >= pos0]
        if self.fp8:
            sc = np.asarray(scales, np.float32).reshape(-1, 2)
            if sc.shape[0] != len(started):
                raise PoolError("INVALID", "one scale pair per started block")
            for j, s in zip(started, sc):
                self.bscale[t][j] = (float(s[0]), float(s[1]))
        elif scales is not None:
            raise PoolError("INVALID", "scales only for fp8 pools")
        self._set_runs(t, pos0, pos0 + n, k, v, 0)

    def _set_runs(self, t, lo, hi, ksrc, vsrc, src_lo):
        out = []
        for r in self.runs[t]:
            a, b, rk, rv, rs = r
            if b <= lo or a >= hi:
                out.append(r)
                continue
            if a < lo:
                out.append([a, lo, rk, rv, rs])
            if b > hi:
                out.append([hi, b, rk, rv, rs + (hi - a)])
        out.append([lo, hi, ksrc, vsrc, src_lo])
        out.sort(key=lambda r: r[0])
        self.runs[t] = out

    # --------------------------------------------------------------- fork --
    def fork(self, parents, children):
        parents = [int(p) for p in parents]
        children = [int(c) for c in children]
        if len(parents) != len(children):
            raise PoolError("INVALID", "parents and children differ in length")
        self._check_ids(children, "child")
        for p in parents:
            if not (0 <= p < self.max_traces):
                raise PoolError("INVALID", "parent id out of range")
        cset = set(children)
        for p, c in zip(parents, children):
            if self.seq_len[c] != 0 or self.table[c]:
                raise PoolError("INVALID", f"child slot {c} is not empty")
            if p in cset:
                raise PoolError("INVALID", "a parent is also a child")
            if self.seq_len[p] == 0:
                raise PoolError("INVALID", f"parent {p} is empty")
        need = sum(1 for p in parents if self.seq_len[p] % self.BS)
        if need > len(self.free):
            raise PoolError("OUT_OF_BLOCKS", f"need {need}, free {len(self.free)}")
        for p, c in zip(parents, children):
            L = self.seq_len[p]
            full = L // self.BS
            for j in range(full):
                b = self.table[p][j]
                self.refcount[b] += 1
                self.table[c].append(b)
            self.bscale[c] = list(self.bscale[p][:self._nblocks(L)])
            if L % self.BS:
                b = self._take_block()
                self.refcount[b] = 1
                self.table[c].append(b)
            self.seq_len[c] = L
            self.runs[c] = [list(r) for r in self.runs[p]]

    # --------------------------------------------------------------- free --
    def free_traces(self, ids):
        ids = [int(t) for t in ids]
        self._check_ids(ids)
        for t in ids:
            if self.seq_len[t] == 0 and not self.table[t]:
                raise PoolError("INVALID", f"trace {t} is already empty")
        for t in ids:
            for b in self.table[t]:
                self.refcount[b] -= 1
                assert self.refcount[b] >= 0
                if self.refcount[b] == 0:
                    heapq.heappush(self.free, b)
            self.table[t] = []
            self.bscale[t] = []
            self.runs[t] = []
            self.seq_len[t] = 0

    # ------------------------------------------------------------- decode --
    def append(self, ids, k_new, v_new):
        """One decode step's append: k_new, v_new are codes [n][Hkv][D] in list order."""
        ids = [int(t) for t in ids]
        self._check_ids(ids)
        for t in ids:
            if self.seq_len[t] == 0:
                raise PoolError("INVALID", f"trace {t} is empty")
            if self._nblocks(self.seq_len[t] + 1) > self.max_blocks:
                raise PoolError("INVALID", "trace exceeds max_blocks_per_trace")
        need = sum(1 for t in ids if self.seq_len[t] % self.BS == 0)
        if need > len(self.free):
            raise PoolError("OUT_OF_BLOCKS", f"need {need}, free {len(self.free)}")
        for i, t in enumerate(ids):
            L = self.seq_len[t]
            self._grow(t, 1, (self.append_scale, self.append_scale))
            self.runs[t].append([L, L + 1, k_new, v_new, i])

    def append_quantised(self, ids, k_bf16, v_bf16):
        """A decode step's append from bf16 K/V (bit patterns [n][Hkv][D], list
        order).  A bf16 pool stores them as they are.  An fp8 pool quantises
        each token with the scale of the block it lands in: the block's own
        (K, V) scales, or append_scale for a block the step opens."""
        if not self.fp8:
            return self.append(ids, k_bf16, v_bf16)
        ids = [int(t) for t in ids]
        kx, vx = bf16_to_f64(k_bf16), bf16_to_f64(v_bf16)
        kc = np.empty(kx.shape, np.uint8)
        vc = np.empty(vx.shape, np.uint8)
        for i, t in enumerate(ids):
            L = self.seq_len[t]
            sk, sv = (self.append_scale, self.append_scale) if L % self.BS == 0 else self.bscale[t][L // self.BS]
            kc[i] = quantise_e4m3fn(kx[i], sk)
            vc[i] = quantise_e4m3fn(vx[i], sv)
        self.append(ids, kc, vc)
        return kc, vc

    # -------------------------------------------------------- materialise --
    def materialise(self, t: int):
        """K, V of trace t as fp64 [L][Hkv][D] (codes decoded, scales applied)."""
        L = self.seq_len[t]
        K = np.full((L, self.Hkv, self.D), np.nan)
        V = np.full((L, self.Hkv, self.D), np.nan)
        for a, b, ks, vs, s0 in self.runs[t]:
            K[a:b] = decode(np.asarray(_resolve(ks))[s0:s0 + b - a], self.kv_dtype)
            V[a:b] = decode(np.asarray(_resolve(vs))[s0:s0 + b - a], self.kv_dtype)
        if self.fp8:
            sk = np.repeat(np.array([s[0] for s in self.bscale[t]], np.float64), self.BS)[:L]
            sv = np.repeat(np.array([s[1] for s in self.bscale[t]], np.float64), self.BS)[:L]
            K *= sk[:, None, None]
            V *= sv[:, None, None]
        return K, V

    # ------------------------------------------------------------ queries --
    def table_array(self, ids=None) -> np.ndarray:
        ids = range(self.max_traces) if ids is None else ids
        out = np.full((len(ids), self.max_blocks), -1, np.int32)
        for i, t in enumerate(ids):
            out[i, :len(self.table[t])] = self.table[t]
        return out

    def check_invariants(self):
        """Refcounts equal reference counts; used + free = all; rows cover lengths."""
        counts = [0] * self.num_blocks
        for t in range(self.max_traces):
            assert self.seq_len[t] == 0 or len(self.table[t]) == self._nblocks(self.seq_len[t])
            for b in self.table[t]:
                counts[b] += 1
        assert counts == self.refcount
        free = set(self.free)
        assert len(free) == len(self.free)
        for b in range(self.num_blocks):
            assert (b in free) == (counts[b] == 0)
