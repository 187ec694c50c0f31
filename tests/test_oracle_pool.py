"""Pins of the oracle's pool model.

* A hand-worked count for the 8-trace workload (512-token prefix, 128-token
  suffixes, one decode step, keep 4 / fork 2).
* Random operation sequences (hypothesis): refcounts equal reference counts,
  used + free = all blocks, rows cover lengths, no row references a free
  block, and every trace's content equals a naive model that stores a full
  private array per trace and copies it at fork.
* Fork equals copy: a forked trace and a trace rebuilt from fresh blocks
  holding a copy of the prefix give bit-identical attention.
* Errors are all-or-nothing.
"""
import math

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle.attention import decode_attention
from oracle.formats import bf16_to_f64
from oracle.pool import PoolError, PoolModel

Hkv, D = 1, 4


def _pool(nb=64, T=6, mb=16, kv="bf16"):
    return PoolModel(num_blocks=nb, n_kv_heads=Hkv, head_dim=D, kv_dtype=kv, max_traces=T,
                     max_blocks_per_trace=mb)


def _codes(rng, n):
    # distinct finite bf16 patterns (exponent field well inside the normal range)
    return (0x3C00 + rng.integers(0, 0x0800, size=(n, Hkv, D))).astype(np.uint16)


def test_hand_worked_config1_counts():
    """8 x 641 tokens: 32 prefix + 64 suffix + 8 tail blocks; keep 4, fork 2 -> 72 used."""
    p = PoolModel(num_blocks=200, n_kv_heads=1, head_dim=1, kv_dtype="bf16", max_traces=8,
                  max_blocks_per_trace=64)
    z = lambda n: np.zeros((n, 1, 1), np.uint16)  # noqa: E731
    p.alloc([0], [512])
    p.write(0, 0, z(512), z(512))
    p.fork([0] * 7, list(range(1, 8)))
    p.alloc(list(range(8)), [128] * 8)
    for t in range(8):
        p.write(t, 512, z(128), z(128))
    p.append(list(range(8)), z(8), z(8))
    assert p.used_blocks() == 104
    prefix = p.table[0][:32]
    assert all(p.refcount[b] == 8 for b in prefix)
    p.free_traces([1, 3, 5, 7])
    assert p.used_blocks() == 104 - 36
    p.fork([0, 2, 4, 6], [1, 3, 5, 7])
    assert p.used_blocks() == 72
    assert all(p.refcount[b] == 8 for b in prefix)
    for par in (0, 2, 4, 6):
        assert all(p.refcount[b] == 2 for b in p.table[par][32:40])
        assert p.refcount[p.table[par][40]] == 1
    for ch in (1, 3, 5, 7):
        assert p.refcount[p.table[ch][40]] == 1 and p.seq_len[ch] == 641
    p.check_invariants()


def test_lowest_free_first_and_list_order():
    p = _pool()
    p.alloc([2, 0], [20, 5])            # trace 2 takes blocks 0,1; trace 0 takes 2
    assert p.table[2] == [0, 1] and p.table[0] == [2]
    p.free_traces([2])
    p.alloc([1], [33])                  # blocks 0, 1, then 3
    assert p.table[1] == [0, 1, 3]


@st.composite
def op_sequences(draw):
    return draw(st.lists(st.tuples(st.integers(0, 4), st.integers(0, 5), st.integers(0, 5),
                                   st.integers(1, 40)), min_size=1, max_size=40))


@settings(max_examples=150, deadline=None)
@given(op_sequences(), st.integers(0, 2 ** 31 - 1))
def test_random_operations_keep_invariants_and_content(ops, seed):
    rng = np.random.default_rng(seed)
    p = _pool()
    naive = {t: np.zeros((0, Hkv, D), np.uint16) for t in range(6)}
    for kind, a, b, n in ops:
        try:
            if kind == 0:
                new = _codes(rng, n)
                L = p.seq_len[a]
                p.alloc([a], [n])
                p.write(a, L, new, new.copy())
                naive[a] = np.concatenate([naive[a], new])
            elif kind == 1 and a != b:
                p.fork([a], [b])
                naive[b] = naive[a].copy()
            elif kind == 2:
                p.free_traces([a])
                naive[a] = naive[a][:0]
            elif kind == 3:
                live = [t for t in range(6) if p.seq_len[t] > 0]
                new = _codes(rng, len(live))
                p.append(live, new, new.copy())
                for i, t in enumerate(live):
                    naive[t] = np.concatenate([naive[t], new[i:i + 1]])
            elif kind == 4 and p.seq_len[a] > 0:
                pos = int(rng.integers(0, p.seq_len[a]))
                new = _codes(rng, 1)
                p.write(a, pos, new, new.copy())
                naive[a] = naive[a].copy()
                naive[a][pos] = new[0]
        except PoolError:
            pass
        p.check_invariants()
        for t in range(6):
            assert p.seq_len[t] == naive[t].shape[0]
            if p.seq_len[t]:
                K, V = p.materialise(t)
                assert np.array_equal(K, bf16_to_f64(naive[t]))
                assert np.array_equal(V, bf16_to_f64(naive[t]))


def test_fork_equals_copy_bit_identical():
    rng = np.random.default_rng(9)
    Hq, Hk, Dd = 8, 2, 128
    p = PoolModel(num_blocks=64, n_kv_heads=Hk, head_dim=Dd, kv_dtype="bf16", max_traces=3,
                  max_blocks_per_trace=32)
    kb = (0x3C00 + rng.integers(0, 0x800, size=(71, Hk, Dd))).astype(np.uint16)
    vb = (0x3C00 + rng.integers(0, 0x800, size=(71, Hk, Dd))).astype(np.uint16)
    p.alloc([0], [71])
    p.write(0, 0, kb, vb)
    p.fork([0], [1])                                   # shares 4 blocks + tail copy
    p.alloc([2], [71])
    p.write(2, 0, kb.copy(), vb.copy())                # private copy
    nk = (0x3C00 + rng.integers(0, 0x800, size=(3, Hk, Dd))).astype(np.uint16)
    p.append([0, 1, 2], nk[[0, 0, 0]], nk[[1, 1, 1]])
    q = rng.standard_normal((Hq, Dd))
    s = 1 / math.sqrt(Dd)
    o1 = decode_attention(q, *p.materialise(1), s)
    o2 = decode_attention(q, *p.materialise(2), s)
    assert np.array_equal(o1, o2)
    assert p.table[1][:4] == p.table[0][:4] and p.table[1][4] != p.table[0][4]


def test_errors_leave_state_unchanged():
    p = _pool(nb=4)
    p.alloc([0], [40])                                  # 3 blocks
    snap = (list(p.free), list(p.refcount), [list(r) for r in p.table], list(p.seq_len))
    with pytest.raises(PoolError) as e:
        p.alloc([1], [40])
    assert e.value.code == "OUT_OF_BLOCKS"
    p.fork([0], [1])                                    # takes the last block (tail of 8)
    with pytest.raises(PoolError) as e:
        p.fork([0], [2])
    assert e.value.code == "OUT_OF_BLOCKS"
    with pytest.raises(PoolError) as e:
        p.write(0, 0, np.zeros((1, Hkv, D), np.uint16), np.zeros((1, Hkv, D), np.uint16))
    assert e.value.code == "SHARED_WRITE"
    with pytest.raises(PoolError) as e:
        p.fork([0], [1])
    assert e.value.code == "INVALID"
    p.free_traces([1])
    with pytest.raises(PoolError) as e:
        p.free_traces([1])
    assert e.value.code == "INVALID"
    assert (list(p.free), list(p.refcount), [list(r) for r in p.table], list(p.seq_len)) == snap


def test_fp8_scales_follow_blocks():
    p = PoolModel(num_blocks=16, n_kv_heads=1, head_dim=2, kv_dtype="fp8_e4m3", max_traces=2,
                  max_blocks_per_trace=8, append_scale=0.5)
    one = np.full((20, 1, 2), 0x38, np.uint8)          # E4M3 code of 1.0
    p.alloc([0], [20])
    p.write(0, 0, one, one, np.array([[2.0, 3.0], [4.0, 5.0]], np.float32))
    p.fork([0], [1])                                    # tail block (4 tokens) copied with scales
    p.append([0, 1], np.full((2, 1, 2), 0x38, np.uint8), np.full((2, 1, 2), 0x38, np.uint8))
    K, V = p.materialise(1)
    assert K[0, 0, 0] == 2.0 and V[0, 0, 0] == 3.0
    assert K[16, 0, 0] == 4.0 and V[19, 0, 1] == 5.0 and K[20, 0, 0] == 4.0
    for t in range(12):
        p.append([0], np.full((1, 1, 2), 0x38, np.uint8), np.full((1, 1, 2), 0x38, np.uint8))
    K, V = p.materialise(0)
    assert K[32, 0, 0] == 0.5 and V[32, 0, 0] == 0.5  # block allocated by a decode step


def test_quantised_append_uses_the_scale_of_the_landing_block():
    """fp8: a token landing in an existing block is quantised with that
    block's (K, V) scales; one that opens a block, with append_scale.  Values
    that are code * scale come back exactly; others within half a code step."""
    p = _pool(kv="fp8_e4m3")
    p.alloc([0], [3])
    p.write(0, 0, np.full((3, Hkv, D), 0x38, np.uint8), np.full((3, Hkv, D), 0x38, np.uint8),
            scales=[[0.5, 0.25]])
    bits = lambda a: (np.asarray(a, np.float32).view(np.uint32) >> 16).astype(np.uint16)
    # K = 1.5 * 0.5 = 0.75, V = 3 * 0.25 = 0.75 exactly; the codes are 1.5 and 3
    kc, vc = p.append_quantised([0], bits(np.full((1, Hkv, D), 0.75)), bits(np.full((1, Hkv, D), 0.75)))
    assert (kc == 0x3C).all() and (vc == 0x44).all()
    K, V = p.materialise(0)
    assert (K[3] == 0.75).all() and (V[3] == 0.75).all()
    # a token that opens a block takes append_scale (2^-6): 0.1 is not a code
    # multiple; the stored value is the nearest multiple of a code
    p.alloc([1], [16])
    p.write(1, 0, np.zeros((16, Hkv, D), np.uint8), np.zeros((16, Hkv, D), np.uint8), scales=[[1.0, 1.0]])
    x = bits(np.full((1, Hkv, D), 0.1))
    p.append_quantised([1], x, x)
    K, V = p.materialise(1)
    assert p.bscale[1][1] == (2.0 ** -6, 2.0 ** -6)
    xv = float(bf16_to_f64(x[0, 0, 0]))
    # 0.1 * 64 = 6.4 lies between the codes 6 and 6.5: 6.5 (step 0.5) is nearer
    assert K[16, 0, 0] == 6.5 * 2.0 ** -6 and abs(K[16, 0, 0] - xv) <= 0.25 * 2.0 ** -6
    # a bf16 pool stores the bits as they are
    q = _pool()
    q.alloc([0], [5])
    q.write(0, 0, np.zeros((5, Hkv, D), np.uint16), np.zeros((5, Hkv, D), np.uint16))
    q.append_quantised([0], x, x)
    assert (q.materialise(0)[0][5] == xv).all()
