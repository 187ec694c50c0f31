"""The workload generator and an oracle replay of whole schedules (CPU)."""
import numpy as np
import pytest

from oracle import run as orun
from workload import CONFIGS, Workload, tiny


def test_generator_is_deterministic_and_keyed():
    a, b = Workload(tiny()), Workload(tiny())
    assert np.array_equal(a.node_kv(3)[0], b.node_kv(3)[0])
    assert np.array_equal(a.step_q(5), b.step_q(5))
    assert not np.array_equal(a.step_q(5), a.step_q(6))


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
def test_tree_shapes_match_configs(cid):
    cfg = CONFIGS[cid]
    wl = Workload(cfg)
    tr = wl.tree
    assert len(tr.leaves) == cfg.n_traces
    assert tr.init_len.max() + cfg.steps <= cfg.ctx_cap
    levels = {}
    for n in tr.nodes:
        levels[n.gen] = levels.get(n.gen, 0) + 1
    assert [levels[g] for g in range(1, len(cfg.gens) + 1)] == list(cfg.gens)
    if cid == 1:
        assert (tr.init_len == 640).all()


def test_config1_replay_block_counts():
    """The hand-worked count through the real generator: 104 blocks, then 72."""
    wl = Workload(CONFIGS[1])
    pool = orun.new_pool(wl, 400)
    orun.apply_setup(pool, wl)
    k, v = wl.step_kv(0)
    ids = list(range(8))
    pool.append(ids, k, v)
    assert pool.used_blocks() == 104
    _, keep, pairs = orun.run_round(pool, wl, 0, ids)
    assert len(keep) == 4 and len(pairs) == 4
    assert pool.used_blocks() == 72
    pool.check_invariants()


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
def test_tiny_schedule_replays(kv):
    wl = Workload(tiny(kv))
    pool = orun.new_pool(wl, 2048)
    orun.apply_setup(pool, wl)
    ids = list(range(wl.T))
    rounds = set(wl.rounds_after())
    for s in range(wl.total_steps):
        k, v = wl.step_kv(s)
        pool.append(ids, k, v)
        out = orun.attend(pool, wl, wl.step_q(s), ids[:2])
        assert all(np.isfinite(o).all() for o in out.values())
        if s in rounds:
            orun.run_round(pool, wl, sorted(rounds).index(s), ids)
        pool.check_invariants()
