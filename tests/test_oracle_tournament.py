"""Pins of the oracle's tournament (Alg. 1 Tournament and Schedule, Eqs. 2-3,
Sec. 4.2), chosen so that a dropped case, a ghost miscounted, a pruned trace
branched, or an inheritance mistake fails one of them:

* Case 2 at capacity is a zero-sum swap: bottom K pruned, top K branched,
  N stays C (Eq. 3); the children hold their parents' full blocks.
* Case 1 under capacity fills min(C - N, |B|) slots from the top eligible
  traces and prunes nothing (Eq. 2).
* Eligibility: GenLen counts decode tokens since creation; a child is not a
  parent until it has generated w tokens; pruned traces never branch.
* Decoupled views (Sec. 4.2): an evicted trace stays in the tree view, so
  the next round is a Case 2 swap rather than a Case 1 refill; a ghost is
  never a parent and leaves only when it falls into the bottom K.
* The running mean equals the arithmetic mean of the thought scores (its
  definition in Sec. 4.1); a child inherits (s_bar, n).
* Eviction takes the running trace of lowest s_bar (Alg. 1 Schedule).
* Count conservation of the runtime example (App. A.5): 256 roots + 1,339
  branches - 1,083 prunes - 256 completions = 256 = C alive; the model's
  counters obey alive = roots + branches - prunes - completions in a random
  run with completions, evictions and both cases.
"""
import random

import numpy as np
import pytest

from oracle.pool import PoolModel
from oracle.tournament import TournamentModel


def _model(T=8, nb=256, mb=32):
    p = PoolModel(num_blocks=nb, n_kv_heads=1, head_dim=1, kv_dtype="bf16", max_traces=T,
                  max_blocks_per_trace=mb)
    return TournamentModel(p)


def _start(m, ids, lengths):
    m.pool.alloc(ids, lengths)


def _scores(m, ids, vals):
    for t, v in zip(ids, vals):
        m.score_update([t], [v])


def test_case2_is_a_zero_sum_swap():
    m = _model(T=6)
    ids = list(range(6))
    _start(m, ids, [40, 33, 17, 64, 5, 50])
    m.decoded(ids)
    _scores(m, ids, [0.5, 0.9, 0.1, 0.7, 0.3, 0.6])
    r = m.tournament(capacity=6, swap_k=2, warmup=0)
    assert r.case == 2 and r.n_active == 6
    assert r.ranked == [1, 3, 5, 0, 4, 2]
    assert r.pruned == [2, 4]                       # bottom K, ascending
    assert r.pairs == [(2, 1), (4, 3)]              # lowest vacant slots, parents in rank order
    assert len(m.tree_view()) == 6
    for c, p in r.pairs:
        full = m.pool.seq_len[p] // 16
        assert m.pool.table[c][:full] == m.pool.table[p][:full]
        assert m.pool.seq_len[c] == m.pool.seq_len[p]
        assert (m.sbar[c], m.nsc[c], m.gen[c]) == (m.sbar[p], m.nsc[p], 0)
    m.pool.check_invariants()


def test_case1_fills_from_the_top_eligible():
    m = _model(T=10)
    ids = [0, 1, 2, 3, 4, 5]
    _start(m, ids, [20] * 6)
    m.decoded(ids)
    _scores(m, ids, [0.2, 0.8, 0.4, 0.9, 0.1, 0.6])
    r = m.tournament(capacity=8, swap_k=3, warmup=0)
    assert r.case == 1 and r.pruned == []
    assert r.pairs == [(6, 3), (7, 1)]              # C - N = 2 children of the top two
    assert len(m.tree_view()) == 8


def test_eligibility_counts_generated_tokens_only():
    m = _model(T=6)
    _start(m, [0, 1, 2, 3], [100, 100, 100, 100])   # prompt writes do not count
    for _ in range(3):
        m.decoded([0, 1, 2, 3])
    m.decoded([2])                                  # trace 2 has generated 4 tokens
    _scores(m, [0, 1, 2, 3], [0.9, 0.8, 0.7, 0.1])
    r = m.tournament(capacity=6, swap_k=1, warmup=4)
    assert r.case == 1 and r.pairs == [(4, 2)]      # 0 and 1 rank higher but are not eligible
    # the child starts at GenLen 0: not a parent until it has generated w tokens
    m.score_update([4], [1.0])                      # now the best-scored trace
    r = m.tournament(capacity=6, swap_k=1, warmup=4)
    assert r.pairs == [(5, 2)]


def test_pruned_traces_never_branch():
    m = _model(T=4)
    ids = [0, 1, 2, 3]
    _start(m, ids, [10] * 4)
    m.decoded([2, 3])                               # only the bottom two are eligible
    _scores(m, ids, [0.9, 0.8, 0.2, 0.1])
    r = m.tournament(capacity=4, swap_k=2, warmup=1)
    assert r.case == 2 and r.pruned == [2, 3] and r.pairs == []
    assert len(m.tree_view()) == 2                  # not zero-sum: next round refills (Case 1)
    m.decoded([0, 1])
    r = m.tournament(capacity=4, swap_k=2, warmup=1)
    assert r.case == 1 and r.pairs == [(2, 0), (3, 1)]


def test_ghosts_keep_capacity_and_rank():
    m = _model(T=6)
    ids = list(range(5))
    _start(m, ids, [30] * 5)
    m.decoded(ids)
    _scores(m, ids, [0.5, 0.95, 0.3, 0.7, 0.6])
    v = m.evict(m.scheduler_view())
    assert v == 2 and m.ghost[2] and m.pool.seq_len[2] == 0
    assert len(m.tree_view()) == 5 and len(m.scheduler_view()) == 4
    # the tree view is still at capacity: a Case 2 swap, which prunes the ghost
    r = m.tournament(capacity=5, swap_k=1, warmup=0)
    assert r.case == 2 and r.pruned == [2] and r.pairs == [(2, 1)]
    # a high-scoring ghost stays and is never a parent
    v = m.evict([1])
    assert v == 1
    r = m.tournament(capacity=5, swap_k=1, warmup=0)
    assert r.case == 2 and 1 not in r.pruned and all(p != 1 for _, p in r.pairs)
    assert r.ranked[0] == 1 and m.ghost[1]


def test_without_ghosts_the_same_run_would_refill():
    """The failure mode Sec. 4.2 describes: counting only the scheduler view."""
    m = _model(T=6)
    ids = list(range(5))
    _start(m, ids, [30] * 5)
    m.decoded(ids)
    _scores(m, ids, [0.5, 0.95, 0.3, 0.7, 0.6])
    m.evict(m.scheduler_view())
    m.ghost[2] = False                              # a model that forgets the ghost
    r = m.tournament(capacity=5, swap_k=1, warmup=0)
    assert r.case == 1 and r.pruned == []


def test_running_mean_and_inheritance():
    rng = np.random.default_rng(3)
    m = _model(T=4)
    _start(m, [0], [25])
    xs = rng.random(37)
    for x in xs:
        m.score_update([0], [x])
    assert m.nsc[0] == 37 and abs(m.sbar[0] - float(np.mean(xs))) < 1e-12
    m.decoded([0])
    m.tournament(capacity=2, swap_k=1, warmup=0)    # Case 1: one child of trace 0
    assert (m.sbar[1], m.nsc[1]) == (m.sbar[0], 37)
    m.score_update([1], [0.0])
    assert abs(m.sbar[1] - float(np.sum(xs)) / 38) < 1e-12


def test_eviction_takes_the_lowest_score_higher_id_on_ties():
    m = _model(T=5)
    ids = list(range(5))
    _start(m, ids, [8] * 5)
    _scores(m, ids, [0.4, 0.2, 0.9, 0.2, 0.5])
    assert m.evict([0, 1, 2, 3, 4]) == 3
    assert m.evict([0, 1, 2, 4]) == 1


def test_random_run_conserves_counts():
    rnd = random.Random(7)
    T, C, K = 24, 16, 4
    m = _model(T=T, nb=4096, mb=64)
    ids = list(range(C))
    _start(m, ids, [rnd.randint(1, 40) for _ in ids])
    roots = C
    for step in range(300):
        live = m.scheduler_view()
        if not live:
            break
        m.pool.alloc(live, [1] * len(live))
        m.decoded(live)
        if step % 7 == 3 and len(live) > 2:
            m.evict(live)
        if step % 11 == 5:
            m.complete([rnd.choice(m.scheduler_view())])
        if step % 5 == 4:
            live = m.scheduler_view()
            m.score_update(live, [rnd.random() for _ in live])
            n_before = len(m.tree_view())
            r = m.tournament(capacity=C, swap_k=K, warmup=6)
            assert r.n_active == n_before
            assert len(m.tree_view()) == n_before - len(r.pruned) + len(r.pairs)
            assert len(m.tree_view()) <= C
            assert not set(p for _, p in r.pairs) & set(r.pruned)
        m.pool.check_invariants()
    alive = len(m.tree_view())
    assert alive == roots + m.branches - m.prunes - m.completions
    assert m.branches > 0 and m.prunes > 0 and m.completions > 0
