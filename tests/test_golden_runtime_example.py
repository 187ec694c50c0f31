"""Pins from the paper's runtime example (App. A.5), read from
tests/golden/runtime_example_app_a5.json: the tournament tree's counts and
the inheritance of the traces it follows, replayed on the oracle's pool and
tournament models."""
from oracle.pool import PoolModel
from oracle.tournament import TournamentModel
from tests._runtime_example import BS, expected_lengths, load, schedule


def test_tree_counts():
    g = load()
    # every node is a root or a branch; a branch fills the slot of a pruned
    # or completed trace (zero-sum), so the population ends at capacity
    assert g["tree_nodes"] == g["roots"] + g["branches"]
    assert g["branches"] == g["pruned"] + g["completed"]
    assert g["roots"] + g["branches"] - g["pruned"] - g["completed"] == g["capacity"]
    assert g["roots"] == g["capacity"]


def _replay(g):
    pool = PoolModel(num_blocks=2600, n_kv_heads=1, head_dim=128, kv_dtype="bf16", max_traces=3,
                     max_blocks_per_trace=2200)
    m = TournamentModel(pool)
    snaps = {}
    for op, a, b in schedule(g):
        if op == "alloc":
            pool.alloc(a, b)
            for t, n in zip(a, b):
                for _ in range(n):
                    m.decoded([t])
        else:
            before = list(pool.refcount)
            pool.fork(a, b)
            snaps[b[0]] = ([list(r) for r in pool.table], list(pool.refcount), before)
        pool.check_invariants()
    return pool, m, snaps


def test_children_inherit_the_parents_context():
    g = load()
    pool, m, snaps = _replay(g)
    p, b = g["tau_p"], g["tau_B"]
    for child, parent, inherited in ((1, 0, p["inherited_tokens"]), (2, 1, b["inherited_tokens"])):
        table, ref, before = snaps[child]
        full = inherited // BS
        # the child's row starts with the parent's full blocks, each with one
        # more reference ...
        assert table[child][:full] == table[parent][:full]
        assert all(ref[x] == before[x] + 1 for x in table[child][:full])
        # ... and its partial last block is a private copy
        assert inherited % BS != 0 and len(table[child]) == full + 1
        assert table[child][full] != table[parent][full] and ref[table[child][full]] == 1
    # lengths at the end: inherited + generated
    for t, L in expected_lengths(g).items():
        assert pool.seq_len[t] == L
    # the founder's first full blocks stay shared by all three traces
    assert all(pool.refcount[x] == 3 for x in pool.table[0][:p["inherited_tokens"] // BS])


def test_warmup_eligibility_of_the_founder():
    """GenLen counts a trace's own tokens only: the root had generated 13,934
    >= w when it branched; tau_p starts at 0 and is eligible to branch once
    it has generated w of its own, which it had when tau_B was branched."""
    g = load()
    w, p, b = g["warmup_tokens"], g["tau_p"], g["tau_B"]
    assert p["created_at_step"] >= w
    pool = PoolModel(num_blocks=2600, n_kv_heads=1, head_dim=128, kv_dtype="bf16", max_traces=3,
                     max_blocks_per_trace=2200)
    m = TournamentModel(pool)
    ops = schedule(g)
    # root generates, then branches tau_p
    pool.alloc(*ops[0][1:])
    for _ in range(p["created_at_step"]):
        m.decoded([0])
    assert m.eligible(0, w)
    pool.fork(*ops[1][1:])
    assert not m.eligible(1, w) and m.gen[1] == 0
    before_b = b["inherited_tokens"] - p["inherited_tokens"]
    pool.alloc(*ops[2][1:])
    for i in range(before_b):
        m.decoded([1])
        assert m.eligible(1, w) == (i + 1 >= w)
    assert m.eligible(1, w)
