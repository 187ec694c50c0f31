"""GPU edge cases through the C ABI: exhaustive fp8 codes, error paths that
must leave the pool unchanged, selection ties, determinism, fork vs copy,
plan splitting, empty calls."""
import math

import numpy as np
import pytest
import torch

from _parity import assert_attn_close
from oracle.attention import decode_attention
from oracle.formats import bf16_to_f64, e4m3fn_to_f64
from oracle.probe import rank
from paper_2608_08020_amd import gambit
from paper_2608_08020_amd.gambit import GambitError, Pool
from workload.generate import to_bf16_bits

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _bf16(x: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(torch.bfloat16).to(DEV)


def test_all_fp8_codes_decode_exactly():
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], np.uint8)
    T, Hkv, Hq = len(codes), 1, 1
    p = Pool(num_blocks=T + 8, num_q_heads=Hq, num_kv_heads=Hkv, max_traces=T,
             max_blocks_per_trace=2, kv_dtype="fp8_e4m3")
    ids = np.arange(T)
    p.kv_alloc(ids, np.ones(T))
    zeros = torch.zeros((1, Hkv, 128), dtype=torch.uint8, device=DEV)
    for t, c in enumerate(codes):
        v = torch.full((1, Hkv, 128), int(c), dtype=torch.uint8, device=DEV)
        p.kv_write(t, 0, zeros, v, np.array([[1.0, 1.0]], np.float32))
    q = torch.zeros((T, Hq, 128), dtype=torch.bfloat16, device=DEV)
    knew = torch.zeros((T, Hkv, 128), dtype=torch.uint8, device=DEV)
    out = p.decode_attn(ids, q, knew, knew, out_dtype=torch.float32)
    # both tokens score 0: o = (decode(code) + 0) / 2 exactly
    want = e4m3fn_to_f64(codes) / 2
    got = out[:, 0, :].cpu().numpy().astype(np.float64)
    assert (got == want[:, None]).all()
    p.pool_check()


def test_second_token_equals_mean_and_first_decode():
    """Two-token context with equal keys gives the mean of the two values."""
    p = Pool(num_blocks=8, num_q_heads=8, num_kv_heads=2, max_traces=2, max_blocks_per_trace=4)
    rng = np.random.default_rng(0)
    k0 = _bf16(np.ones((1, 2, 128)))
    v0 = _bf16(rng.standard_normal((1, 2, 128)))
    p.kv_alloc([0], [1])
    p.kv_write(0, 0, k0, v0)
    q = _bf16(rng.standard_normal((1, 8, 128)))
    v1 = _bf16(rng.standard_normal((1, 2, 128)))
    out = p.decode_attn([0], q, k0, v1, out_dtype=torch.float32).cpu().numpy()[0]
    want = (v0.float().cpu().numpy()[0] + v1.float().cpu().numpy()[0]) / 2
    for h in range(8):
        assert np.abs(out[h] - want[h // 4]).max() <= 1e-6


def test_errors_leave_pool_unchanged():
    p = Pool(num_blocks=6, num_q_heads=4, num_kv_heads=1, max_traces=4, max_blocks_per_trace=8)
    x = torch.zeros((40, 1, 128), dtype=torch.bfloat16, device=DEV)
    p.kv_alloc([0], [40])                                    # 3 blocks
    p.kv_write(0, 0, x, x)
    cases = [
        ("OUT_OF_BLOCKS", lambda: p.kv_alloc([1], [64])),
        ("INVALID", lambda: p.kv_alloc([0, 0], [1, 1])),
        ("INVALID", lambda: p.kv_alloc([9], [1])),
        ("INVALID", lambda: p.kv_alloc([1], [200])),         # exceeds max_blocks_per_trace
        ("INVALID", lambda: p.kv_write(0, 30, x[:20], x[:20])),
        ("INVALID", lambda: p.kv_fork([1], [2])),            # empty parent
        ("INVALID", lambda: p.kv_free([3])),                 # already empty
        ("INVALID", lambda: p.decode_attn([1], torch.zeros((1, 4, 128), dtype=torch.bfloat16, device=DEV),
                                          x[:1], x[:1])),    # empty trace
    ]
    for code, fn in cases:
        with pytest.raises(GambitError) as e:
            fn()
        assert e.value.code == code, (code, str(e.value))
        p.pool_check()
    p.kv_fork([0], [1])                                      # takes 1 block (tail of 8)
    with pytest.raises(GambitError) as e:
        p.kv_write(0, 0, x[:1], x[:1])
    assert e.value.code == "SHARED_WRITE"
    with pytest.raises(GambitError) as e:
        p.kv_fork([0], [1])
    assert e.value.code == "INVALID"
    p.kv_alloc([2], [32])                                    # the last 2 blocks
    with pytest.raises(GambitError) as e:
        p.kv_fork([0], [3])
    assert e.value.code == "OUT_OF_BLOCKS"
    with pytest.raises(GambitError) as e:
        p.score_prune_branch([0, 1, 2], torch.zeros((3, 64), dtype=torch.bfloat16, device=DEV),
                             torch.zeros(64, device=DEV), 0.0, 2, 2)   # 1 pruned over 2 parents
    assert e.value.code == "INVALID"
    p.pool_check()
    assert p.free_blocks() == 0


def test_rank_topk_ties_bit_exact():
    rng = np.random.default_rng(1)
    # sizes on both sides of the run-merge sort's limits (runs of 128, at most
    # 1024 keys; the bitonic network beyond), crafted ties
    for n, keep in [(7, 3), (512, 128), (1000, 999), (4096, 17), (33, 33), (1, 1), (64, 10), (128, 64),
                    (129, 1), (256, 256), (1024, 1024), (1025, 500), (2048, 2000)]:
        ids = rng.permutation(n * 3)[:n].astype(np.int32)
        scores = rng.choice(np.array([0.1, 0.5, 0.5000001, 0.9, -2.0], np.float32), size=n)
        got = gambit.rank_topk(torch.from_numpy(ids).to(DEV), torch.from_numpy(scores).to(DEV), keep)
        want = rank(ids, scores.astype(np.float64))[:keep]
        assert got.cpu().numpy().tolist() == want


def test_deterministic_bitwise():
    from paper_2608_08020_amd.runner import PopulationRun
    from workload import Workload, tiny

    outs = []
    for _ in range(2):
        wl = Workload(tiny())
        run = PopulationRun(wl)
        run.setup()
        run.load_steps(range(wl.total_steps))
        run.load_rounds(range(len(wl.rounds_after())))
        res = []
        for s, r in run.schedule():
            res.append(run.decode(s, out_dtype=torch.float32).cpu().numpy())
            if r is not None:
                res.append(np.concatenate([x.cpu().numpy().ravel().view(np.uint32) for x in run.round(r)[1:]]))
        res.append(run.pool.block_table.cpu().numpy())
        outs.append(res)
    for a, b in zip(*outs):
        assert np.array_equal(a.view(np.uint8), b.view(np.uint8))


def test_fork_and_copy_agree():
    rng = np.random.default_rng(2)
    p = Pool(num_blocks=64, num_q_heads=8, num_kv_heads=2, max_traces=3, max_blocks_per_trace=16)
    k = _bf16(rng.standard_normal((71, 2, 128)))
    v = _bf16(rng.standard_normal((71, 2, 128)))
    p.kv_alloc([0], [71])
    p.kv_write(0, 0, k, v)
    p.kv_fork([0], [1])
    p.kv_alloc([2], [71])
    p.kv_write(2, 0, k.clone(), v.clone())
    q = _bf16(np.repeat(rng.standard_normal((1, 8, 128)), 3, axis=0))
    kn = _bf16(np.repeat(rng.standard_normal((1, 2, 128)), 3, axis=0))
    vn = _bf16(np.repeat(rng.standard_normal((1, 2, 128)), 3, axis=0))
    out = p.decode_attn([0, 1, 2], q, kn, vn, out_dtype=torch.float32).cpu().numpy()
    K = np.concatenate([bf16_to_f64(k.cpu().view(torch.int16).numpy().view(np.uint16)),
                        bf16_to_f64(kn[:1].cpu().view(torch.int16).numpy().view(np.uint16))])
    V = np.concatenate([bf16_to_f64(v.cpu().view(torch.int16).numpy().view(np.uint16)),
                        bf16_to_f64(vn[:1].cpu().view(torch.int16).numpy().view(np.uint16))])
    ref = decode_attention(bf16_to_f64(q[0].cpu().view(torch.int16).numpy().view(np.uint16)), K, V,
                           1 / math.sqrt(128))
    for t in range(3):
        assert_attn_close(out[t], ref, f"fork/copy trace {t}")
    tab = p.block_table.cpu().numpy()
    assert (tab[1, :4] == tab[0, :4]).all() and tab[1, 4] != tab[0, 4]
    p.pool_check()


def test_split_limit_grows_chunks_or_reports():
    rng = np.random.default_rng(3)
    p = Pool(num_blocks=600, num_q_heads=4, num_kv_heads=1, max_traces=2, max_blocks_per_trace=300,
             max_splits=1)
    L = 4000
    k = _bf16(rng.standard_normal((L, 1, 128)))
    v = _bf16(rng.standard_normal((L, 1, 128)))
    p.kv_alloc([0], [L])
    p.kv_write(0, 0, k, v)
    q = _bf16(rng.standard_normal((1, 4, 128)))
    kn = _bf16(rng.standard_normal((1, 1, 128)))
    out = p.decode_attn([0], q, kn, kn, out_dtype=torch.float32).cpu().numpy()[0]
    assert p.plan_stats([0]).max_splits_used == 1
    K = np.concatenate([k.float().cpu().numpy(), kn.float().cpu().numpy()]).astype(np.float64)
    V = np.concatenate([v.float().cpu().numpy(), kn.float().cpu().numpy()]).astype(np.float64)
    ref = decode_attention(q[0].float().cpu().numpy().astype(np.float64), K, V, 1 / math.sqrt(128))
    assert_attn_close(out, ref, "one partial per trace")
    # after a fork every trace has a shared run and a private run: two partials
    p.kv_fork([0], [1])
    with pytest.raises(GambitError) as e:
        p.decode_attn([0, 1], q.repeat(2, 1, 1), kn.repeat(2, 1, 1), kn.repeat(2, 1, 1))
    assert e.value.code == "UNSUPPORTED"
    p.pool_check()


def test_empty_calls_are_no_ops():
    p = Pool(num_blocks=4, num_q_heads=4, num_kv_heads=1, max_traces=2, max_blocks_per_trace=2)
    z = torch.zeros((0, 4, 128), dtype=torch.bfloat16, device=DEV)
    p.kv_alloc([], [])
    p.kv_free([])
    p.kv_fork([], [])
    p.decode_attn([], z, z[:, :1], z[:, :1])
    p.pool_check()
    assert p.free_blocks() == 4


@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8_e4m3"])
def test_many_blocks_opened_in_one_step(kv_dtype):
    """A decode step whose appends open more blocks than its launch carries
    (the allocator kernel runs first) and steps that open fewer (the attention
    launch claims them), with the trace list out of id order and freed blocks
    interleaved with used ones: tables, refcounts, lengths, scales and
    attention as the pool model gives them."""
    from oracle.pool import PoolModel

    fp8 = kv_dtype == "fp8_e4m3"
    T, Hq, Hkv = 300, 4, 1
    rng = np.random.default_rng(11)
    p = Pool(num_blocks=1200, num_q_heads=Hq, num_kv_heads=Hkv, max_traces=T, max_blocks_per_trace=4,
             kv_dtype=kv_dtype)
    om = PoolModel(num_blocks=1200, n_kv_heads=Hkv, head_dim=128, kv_dtype=kv_dtype, max_traces=T,
                   max_blocks_per_trace=4)

    def codes(n):
        if fp8:
            c = rng.integers(0, 256, size=(n, Hkv, 128)).astype(np.uint8)
            c[(c & 0x7F) == 0x7F] = 0x38  # no NaN codes
            return c
        return to_bf16_bits(rng.standard_normal((n, Hkv, 128)).astype(np.float32))

    def bf16_dev(c):
        return torch.from_numpy(c.view(np.int16)).view(torch.bfloat16).to(DEV)

    def dev(c):
        return torch.from_numpy(c).to(DEV) if fp8 else bf16_dev(c)

    def fill(t, L):
        p.kv_alloc([t], [L])
        om.alloc([t], [L])
        k, v = codes(L), codes(L)
        sc = np.full(((L + 15) // 16, 2), 0.5 + t / T, np.float32) if fp8 else None
        p.kv_write(t, 0, dev(k), dev(v), sc)
        om.write(t, 0, k, v, sc)

    for t in range(T):
        fill(t, 16 if t < 270 else 7)

    def step(ids):
        n = len(ids)
        q = to_bf16_bits(rng.standard_normal((n, Hq, 128)).astype(np.float32))
        kn, vn = codes(n), codes(n)
        out = p.decode_attn(ids, bf16_dev(q), dev(kn), dev(vn), out_dtype=torch.float32).cpu().numpy()
        om.append(ids, kn, vn)
        for i in list(range(0, n, 37)) + [n - 1]:
            K, V = om.materialise(int(ids[i]))
            ref = decode_attention(bf16_to_f64(q[i]), K, V, 1 / math.sqrt(128))
            assert_attn_close(out[i], ref, f"trace {ids[i]} (list position {i})")
        assert p.seq_len.cpu().numpy().tolist() == om.seq_len
        assert np.array_equal(p.block_table.cpu().numpy(), om.table_array())
        assert p.refcount.cpu().numpy().tolist() == om.refcount
        if fp8:
            sc = p.kv_scale.cpu().numpy()
            for t in ids:
                assert [tuple(sc[b]) for b in om.table[t]] == om.bscale[t], t
        p.pool_check()

    step(rng.permutation(T))        # 270 blocks opened: more than one launch carries
    step(rng.permutation(T))        # none opened
    for t in range(0, 200, 2):      # frees 100 traces' blocks between used ones
        p.kv_free([t])
        om.free_traces([t])
    for t in range(0, 200, 2):
        fill(t, 32)
    step(rng.permutation(T))        # 100 opened, claimed by the attention launch
    step(rng.permutation(T)[:150])  # a partial list


@pytest.mark.parametrize("opening", [256, 257])
def test_launch_argument_capacity_boundary(opening):
    """Exactly as many new blocks as one launch carries (256: claimed by the
    attention launch) and one more (257: the allocator kernel runs first)."""
    from oracle.pool import PoolModel

    T, Hq, Hkv = 300, 4, 1
    rng = np.random.default_rng(12 + opening)
    p = Pool(num_blocks=800, num_q_heads=Hq, num_kv_heads=Hkv, max_traces=T, max_blocks_per_trace=3)
    om = PoolModel(num_blocks=800, n_kv_heads=Hkv, head_dim=128, kv_dtype="bf16", max_traces=T,
                   max_blocks_per_trace=3)
    for t in range(T):
        L = 16 if t < opening else 9
        kv = to_bf16_bits(rng.standard_normal((L, Hkv, 128)).astype(np.float32))
        dev = torch.from_numpy(kv.view(np.int16)).view(torch.bfloat16).to(DEV)
        p.kv_alloc([t], [L])
        p.kv_write(t, 0, dev, dev)
        om.alloc([t], [L])
        om.write(t, 0, kv, kv)
    ids = rng.permutation(T)
    q = to_bf16_bits(rng.standard_normal((T, Hq, 128)).astype(np.float32))
    kn = to_bf16_bits(rng.standard_normal((T, Hkv, 128)).astype(np.float32))
    bf = lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(DEV)  # noqa: E731
    out = p.decode_attn(ids, bf(q), bf(kn), bf(kn), out_dtype=torch.float32).cpu().numpy()
    om.append(ids, kn, kn)
    assert np.array_equal(p.block_table.cpu().numpy(), om.table_array())
    assert p.seq_len.cpu().numpy().tolist() == om.seq_len
    for i in (0, 99, T - 1):
        K, V = om.materialise(int(ids[i]))
        ref = decode_attention(bf16_to_f64(q[i]), K, V, 1 / math.sqrt(128))
        assert_attn_close(out[i], ref, f"trace {ids[i]} (list position {i})")
    p.pool_check()
