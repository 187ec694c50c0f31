"""The full thought-level tournament of Alg. 1 over the pool model.  Test
infrastructure only.

Per trace slot the model keeps what Alg. 1 reads:

* the running mean score s_bar and the number n of scored thoughts
  (Alg. 1 Generate: s_bar <- s_bar + (f(h_n) - s_bar) / n when a trace
  completes thought n; Sec. 4.1 defines s_bar as the mean of the per-thought
  scores);
* GenLen, the tokens a trace has generated since its own creation (the
  eligibility test GenLen >= w of Alg. 1 Tournament and Sec. 4.1); decode
  steps generate, prompt writes do not;
* the ghost flag of the decoupled views (Sec. 4.2): a trace the scheduler
  evicted under memory pressure (Alg. 1 Schedule: the running trace of
  lowest s_bar) holds no KV and generates nothing, but stays in the tree
  view, so it counts towards the capacity check and keeps its rank.

A tournament (Alg. 1 Tournament, Eqs. 2-3) ranks the tree view (live and
ghost traces) by s_bar, highest first, ties to the lower slot id, then

* Case 1, N < C: branch the top min(C - N, |B|) eligible traces (Eq. 2);
* Case 2, N >= C: prune the bottom K, then branch the top K eligible traces
  that were not pruned (Eq. 3; the swap is zero-sum when K of them exist).

Readings where the paper is silent (each also listed in the design notes):
eligible = live (not a ghost) and GenLen >= w, and in Case 2 not among the
pruned; N > C is handled as Case 2; a child inherits its parent's (s_bar, n)
(the child's trace is the parent's prefix plus its own thoughts) and starts
with GenLen 0; pruned slots are freed in ascending id order before any
fork; children take the lowest vacant slot ids in ascending order, one per
parent in rank order (App. A.5: each branching event is a 1-to-1 split in
which the parent continues); the eviction victim among equal scores is the
higher id (the trace ranked last); completing a trace removes it from both
views.
"""
from __future__ import annotations

from dataclasses import dataclass, field

from .pool import PoolError, PoolModel


@dataclass
class RoundResult:
    case: int                       # 1 or 2 (0: empty tree view, nothing to do)
    n_active: int                   # N, the tree view's size before the round
    ranked: list                    # the tree view by (s_bar desc, id asc)
    pruned: list = field(default_factory=list)   # ascending ids
    pairs: list = field(default_factory=list)    # [(child, parent)] in branch order


class TournamentModel:
    """Tree view, scheduler view and per-trace scores over a PoolModel."""

    def __init__(self, pool: PoolModel):
        self.pool = pool
        T = pool.max_traces
        self.sbar = [0.0] * T
        self.nsc = [0] * T
        self.gen = [0] * T
        self.ghost = [False] * T
        self.branches = 0
        self.prunes = 0
        self.completions = 0

    # ------------------------------------------------------------ views --
    def live(self, t: int) -> bool:
        """Scheduler view: the trace holds KV blocks."""
        return self.pool.seq_len[t] > 0

    def tree_view(self) -> list:
        return [t for t in range(self.pool.max_traces) if self.live(t) or self.ghost[t]]

    def scheduler_view(self) -> list:
        return [t for t in range(self.pool.max_traces) if self.live(t)]

    def eligible(self, t: int, w: int) -> bool:
        return self.live(t) and not self.ghost[t] and self.gen[t] >= w

    def rank(self, ids) -> list:
        return sorted(ids, key=lambda t: (-self.sbar[t], t))

    def _reset(self, t: int):
        self.sbar[t], self.nsc[t], self.gen[t], self.ghost[t] = 0.0, 0, 0, False

    # ---------------------------------------------------------- generate --
    def decoded(self, ids):
        """A decode step generated one token for each listed trace."""
        for t in ids:
            self.gen[t] += 1

    def score_update(self, ids, f):
        """The listed traces completed a thought scored f (Alg. 1 Generate)."""
        for t, x in zip(ids, f):
            if not self.live(t):
                raise PoolError("INVALID", f"trace {t} is not running")
            self.nsc[t] += 1
            self.sbar[t] += (float(x) - self.sbar[t]) / self.nsc[t]

    # ---------------------------------------------------------- schedule --
    def evict(self, candidates) -> int:
        """Memory pressure: the listed running trace of lowest s_bar becomes a
        ghost (Alg. 1 Schedule; Sec. 4.2).  Returns its id."""
        cand = [int(t) for t in candidates]
        if not cand or any(not self.live(t) for t in cand):
            raise PoolError("INVALID", "eviction candidates must be running traces")
        victim = self.rank(cand)[-1]
        self.pool.free_traces([victim])
        self.ghost[victim] = True
        self.gen[victim] = 0
        return victim

    def complete(self, ids):
        """Completed traces leave both views (Alg. 1: moved to F)."""
        ids = [int(t) for t in ids]
        self.pool.free_traces(ids)
        for t in ids:
            self._reset(t)
        self.completions += len(ids)

    # -------------------------------------------------------- tournament --
    def tournament(self, capacity: int, swap_k: int, warmup: int) -> RoundResult:
        act = self.tree_view()
        N = len(act)
        ranked = self.rank(act)
        if N == 0:
            return RoundResult(0, 0, [])
        if N < capacity:                               # Case 1 (Eq. 2)
            case, pruned = 1, []
            B = [t for t in ranked if self.eligible(t, warmup)]
            m = min(capacity - N, len(B))
        else:                                          # Case 2 (Eq. 3)
            case = 2
            nprune = min(swap_k, N)
            pruned = sorted(ranked[N - nprune:])
            gone = set(pruned)
            B = [t for t in ranked if t not in gone and self.eligible(t, warmup)]
            m = min(swap_k, len(B))
        parents = B[:m]
        # prune: free the KV of running traces, drop ghosts from the tree view
        running = [t for t in pruned if self.live(t)]
        if running:
            self.pool.free_traces(running)
        for t in pruned:
            self._reset(t)
        self.prunes += len(pruned)
        # branch into the lowest vacant slots
        vacant = [t for t in range(self.pool.max_traces) if not self.live(t) and not self.ghost[t]]
        if len(vacant) < m:
            raise PoolError("INVALID", "fewer vacant slots than children")
        children = vacant[:m]
        if m:
            self.pool.fork(parents, children)
        for c, p in zip(children, parents):
            self.sbar[c], self.nsc[c], self.gen[c], self.ghost[c] = self.sbar[p], self.nsc[p], 0, False
        self.branches += m
        return RoundResult(case, N, ranked, pruned, list(zip(children, parents)))
