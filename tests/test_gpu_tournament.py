"""GPU parity of the full tournament of Alg. 1 (running-mean scores, GenLen
eligibility, Case 1 / Case 2, scheduler eviction into ghosts, completions)
against the oracle, through the C ABI; plus its error paths, which must
leave the pool unchanged.  See _tournament.py for the bars."""
import numpy as np
import pytest
import torch

from _tournament import run
from paper_2608_08020_amd.gambit import GambitError, Pool
from workload.tournament import TOURNAMENT_C256, TOURNAMENT_SMALL

pytestmark = pytest.mark.gpu


def test_small_tournament_run():
    st = run(TOURNAMENT_SMALL, attn_steps={0, 9, 24, 40, 61, 79}, sample=4)
    assert st["case1"] > 0 and st["case2"] > 0 and st["ghosts_pruned"] > 0 and st["attn_checked"] > 0


@pytest.mark.timeout(600)
def test_c256_tournament_run():
    st = run(TOURNAMENT_C256, attn_steps={0, 47, 128, 255}, sample=3)
    assert st["case1"] > 0 and st["case2"] > 0 and st["alive"] == TOURNAMENT_C256.capacity


def _pool():
    p = Pool(num_blocks=64, num_q_heads=4, num_kv_heads=1, max_traces=6, max_blocks_per_trace=8)
    p.kv_alloc([0, 1, 2], [20, 9, 33])
    return p


def test_tournament_errors_change_nothing():
    p = _pool()
    before = (p.block_table.clone(), p.seq_len.clone())
    for args in [(0, 1, 0), (7, 1, 0), (3, -1, 0), (3, 1, -2)]:
        with pytest.raises(GambitError) as e:
            p.tournament(*args)
        assert e.value.code == "INVALID"
    assert torch.equal(p.block_table, before[0]) and torch.equal(p.seq_len, before[1])
    with pytest.raises(GambitError):
        p.evict([0, 4])            # slot 4 is not running
    with pytest.raises(GambitError):
        p.evict([])
    p.pool_check()
    # a ghost: not extendable, not a fork target, not a score or eviction target
    v = p.evict([0, 1, 2])
    assert p.seq_len_of(v) == 0
    for bad in [lambda: p.kv_alloc([v], [4]), lambda: p.kv_fork([2 if v != 2 else 1], [v]),
                lambda: p.evict([v]), lambda: p.kv_free([v])]:
        with pytest.raises(GambitError):
            bad()
    p.pool_check()
    sb, ns, ge, gh = p.trace_state([v])
    assert gh[0] == 1


def test_empty_tree_view_is_a_no_op():
    p = Pool(num_blocks=16, num_q_heads=4, num_kv_heads=1, max_traces=4, max_blocks_per_trace=4)
    case, n, pruned, pairs, _ = p.tournament(2, 1, 0)
    assert (case, n, pruned, pairs) == (0, 0, [], [])
    p.pool_check()
