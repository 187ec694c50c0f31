"""The C-ABI library loads on a machine without a GPU and exports every
entry point include/gambit.h declares; host-only queries work."""
import ctypes
import os
import re

import numpy as np

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    text = open(os.path.join(ROOT, "include", "gambit.h")).read()
    return sorted(set(re.findall(r"^\s*(?:[\w*]+\s+\**)+(gambit_\w+)\s*\(", text, re.M)))


def test_header_declares_the_hot_path_calls():
    names = _declared()
    for want in ["gambit_kv_alloc", "gambit_kv_fork", "gambit_kv_free", "gambit_kv_write",
                 "gambit_decode_attn", "gambit_score_prune_branch", "gambit_pool_create"]:
        assert want in names


def test_library_exports_every_declared_symbol():
    from paper_2608_08020_amd import gambit
    if not os.path.exists(gambit.LIB_PATH):
        pytest.skip("libgambit.so not built")
    L = gambit.lib()
    for name in _declared():
        assert hasattr(L, name), name
    assert set(_declared()) == set(gambit.EXPORTS)


def test_workspace_size_validates_descriptions():
    from paper_2608_08020_amd import gambit
    if not os.path.exists(gambit.LIB_PATH):
        pytest.skip("libgambit.so not built")
    d = gambit.PoolDesc(num_blocks=1000, block_size=16, num_q_heads=32, num_kv_heads=8, head_dim=128,
                        kv_dtype=0, max_traces=64, max_blocks_per_trace=100, max_splits=0, fp8_append_scale=0.0,
                        num_layers=1)
    ok = gambit.workspace_size(d)
    assert ok > 0
    for field, bad in [("head_dim", 64), ("block_size", 32), ("num_q_heads", 12), ("kv_dtype", 7),
                       ("num_blocks", 0), ("num_layers", -1), ("num_layers", 5000)]:
        d2 = gambit.PoolDesc.from_buffer_copy(d)
        setattr(d2, field, bad)
        assert gambit.workspace_size(d2) == 0, field
    # fewer partial slots, less workspace
    d3 = gambit.PoolDesc.from_buffer_copy(d)
    d3.max_splits = 16
    assert 0 < gambit.workspace_size(d3) < ok
    # the merge reads a row's partials one per lane: at most 64
    d3.max_splits = 65
    assert gambit.workspace_size(d3) == 0
    assert gambit.lib().gambit_status_str(-2).decode() == "out of KV blocks"


def test_scorer_workspace_size_validates_descriptions():
    from paper_2608_08020_amd import gambit
    if not os.path.exists(gambit.LIB_PATH):
        pytest.skip("libgambit.so not built")
    L = gambit.lib()
    d = gambit.ScorerDesc(input_dim=4096, d_model=256, n_heads=4, n_layers=2, d_ff=768, max_steps=256,
                          max_traces=512)
    ok = int(L.gambit_scorer_workspace_size(ctypes.byref(d)))
    # the per-slot key / value caches dominate: 512 x 2 layers x 4 heads x 2 x 64 x 256 fp32
    assert ok >= 512 * 2 * 4 * 2 * 64 * 256 * 4
    for field, bad in [("d_model", 200), ("n_heads", 3), ("input_dim", 100), ("input_dim", 192), ("d_ff", 100), ("max_steps", 0),
                       ("max_steps", 9000), ("n_layers", -1), ("max_traces", 0)]:
        d2 = gambit.ScorerDesc.from_buffer_copy(d)
        setattr(d2, field, bad)
        assert int(L.gambit_scorer_workspace_size(ctypes.byref(d2))) == 0, field
    # no layers: no caches
    d3 = gambit.ScorerDesc.from_buffer_copy(d)
    d3.n_layers = 0
    assert 0 < int(L.gambit_scorer_workspace_size(ctypes.byref(d3))) < ok


def test_stream_read_rejects_bad_arguments_without_a_device():
    from paper_2608_08020_amd import gambit
    if not os.path.exists(gambit.LIB_PATH):
        pytest.skip("libgambit.so not built")
    L = gambit.lib()
    fake = ctypes.c_void_p(1 << 20)  # never dereferenced: every call below fails validation
    sink = ctypes.c_void_p(1 << 21)
    bad = [(None, 65536, 0, 1, sink), (fake, 0, 0, 1, sink), (fake, 65536 + 16, 0, 1, sink),
           (fake, 65536, 0, 0, sink), (fake, 65536, 0, 2, sink), (fake, 65536 * 70000, 0, 65536, sink),
           (fake, 65536, 2, 1, sink), (fake, 65536, 0, 1, None), (ctypes.c_void_p((1 << 20) + 4), 65536, 0, 1, sink)]
    for buf, nbytes, nt, grid, snk in bad:
        assert L.gambit_stream_read(buf, nbytes, nt, grid, snk, None) == gambit.ERR_INVALID


def _fake_pool(kv_dtype="bf16", Hq=32, Hkv=8, num_layers=1):
    """A Pool object without a device pool behind it: the binding's argument
    checks run before any library call, so they can be exercised on a
    machine without a GPU (every call below must fail in them)."""
    import torch

    from paper_2608_08020_amd import gambit
    p = gambit.Pool.__new__(gambit.Pool)
    p.kv_dtype, p.Hq, p.Hkv, p.D, p.num_layers = kv_dtype, Hq, Hkv, 128, num_layers
    p.cache_dtype = torch.uint8 if kv_dtype == "fp8_e4m3" else torch.bfloat16
    p.max_traces, p.max_blocks = 16, 8
    p._h = None
    return p


def _raises(fn, match):
    with pytest.raises(ValueError, match=match):
        fn()


def test_binding_checks_every_device_argument():
    """Short or mistyped buffers would be read or written past their end by
    the kernels (the C ABI takes bare pointers), so the binding checks each
    one's dtype and shape first."""
    import torch
    bf, f32, u8, i32 = torch.bfloat16, torch.float32, torch.uint8, torch.int32
    z = lambda *s, dt=bf: torch.zeros(s, dtype=dt)  # noqa: E731
    n = 4
    for kvd, cdt in [("bf16", bf), ("fp8_e4m3", u8)]:
        p = _fake_pool(kvd)
        q, kn, out = z(n, 32, 128), z(n, 8, 128, dt=cdt), z(n, 32, 128, dt=f32)
        ids = list(range(n))
        _raises(lambda: p.decode_attn(ids, q, kn, kn, out=z(n - 1, 32, 128, dt=f32)), "out: expected shape")
        _raises(lambda: p.decode_attn(ids, q, kn, kn, out=z(n, 32, 128, dt=torch.float16)), "out: expected dtype")
        _raises(lambda: p.decode_attn(ids, z(n, 32, 64), kn, kn, out=out), "q: expected shape")
        _raises(lambda: p.decode_attn(ids, q, z(n - 1, 8, 128, dt=cdt), kn, out=out), "k_new: expected shape")
        _raises(lambda: p.decode_attn(ids, q, kn, z(n, 8, 127, dt=cdt), out=out), "v_new: expected shape")
        other = u8 if cdt == bf else bf
        _raises(lambda: p.decode_attn(ids, q, z(n, 8, 128, dt=other), kn, out=out), "k_new: expected dtype")
        _raises(lambda: p.decode_attn(ids, q, kn, kn, out=out), "expected a device tensor")  # all well-formed
        # one layer of a step: new K/V in the cache dtype or bf16 (quantised on append)
        _raises(lambda: p.decode_attn_layer(0, ids, q, z(n, 8, 128, dt=other if cdt == u8 else u8), kn, out=out),
                "k_new: expected dtype")
        _raises(lambda: p.decode_attn_layer(0, ids, q, z(n, 8, 128), z(n - 1, 8, 128), new_dtype="bf16", out=out),
                "v_new: expected shape")
        _raises(lambda: p.decode_attn_layer(0, ids, q, kn, kn, new_dtype="fp16", out=out), "new_dtype")
        # writes: [n][Hkv][D] in the cache dtype; fp8 scales one (K, V) pair per block started
        _raises(lambda: p.kv_write(0, 0, z(20, 8, 128, dt=cdt), z(19, 8, 128, dt=cdt)), "v: expected shape")
        _raises(lambda: p.kv_write(0, 0, z(20, 4, 128, dt=cdt), z(20, 4, 128, dt=cdt)), "k: expected shape")
    p = _fake_pool("fp8_e4m3")
    k20 = z(20, 8, 128, dt=u8)
    _raises(lambda: p.kv_write(0, 0, k20, k20, np.ones((1, 2), np.float32)), "scales: expected shape \\(2, 2\\)")
    _raises(lambda: p.kv_write(0, 10, k20, k20, np.ones((1, 2), np.float32)), "expected a device tensor")  # one block starts in 10..29
    _raises(lambda: p.kv_write(0, 10, k20, k20, np.ones((2, 2), np.float32)), "scales: expected shape \\(1, 2\\)")
    _raises(lambda: _fake_pool("bf16").kv_write(0, 0, z(3, 8, 128), z(3, 8, 128), np.ones((1, 2))), "scales: only fp8")
    # a thought boundary: h [n][Dh] bf16, w [Dh] fp32
    p = _fake_pool()
    _raises(lambda: p.score_prune_branch(range(n), z(n - 1, 64), z(64, dt=f32), 0.0, 2, 2), "h: expected shape")
    _raises(lambda: p.score_prune_branch(range(n), z(n, 64), z(32, dt=f32), 0.0, 2, 2), "w: expected shape")
    _raises(lambda: p.score_prune_branch(range(n), z(n, 64, dt=f32), z(64, dt=f32), 0.0, 2, 2), "h: expected dtype")
    _raises(lambda: p.score_prune_branch(range(n), z(n, 64), z(64, dt=f32), 0.0, 5, 2), "keep")
    _raises(lambda: p.score_update(range(n), z(n - 1, 64), z(64, dt=f32), 0.0), "h: expected")
    _raises(lambda: p.score_update(range(n), z(n, 64), z(63, dt=f32), 0.0), "w: expected shape")
    _raises(lambda: p.record_scores(range(n), z(n - 1, dt=f32)), "f: expected")
    # the stateless calls
    from paper_2608_08020_amd.gambit import mlp_score, rank_topk
    h, w1, b1, w2 = z(n, 256), z(128, 256), z(128, dt=f32), z(128, dt=f32)
    _raises(lambda: mlp_score(h, z(128, 255), b1, w2, 0.0), "w1: expected shape")
    _raises(lambda: mlp_score(h, w1, z(127, dt=f32), w2, 0.0), "b1: expected shape")
    _raises(lambda: mlp_score(h, w1, b1, z(128), 0.0), "w2: expected dtype")
    _raises(lambda: mlp_score(h, w1, b1, w2, 0.0, keep=2), "ids: needed")
    _raises(lambda: mlp_score(h, w1, b1, w2, 0.0, ids=z(n - 1, dt=i32), keep=2), "ids: expected shape")
    _raises(lambda: rank_topk(z(n, dt=i32), z(n - 1, dt=f32), 2), "scores: expected shape")


def test_mlp_workspace_sizes_and_checks():
    """Workspace sizes of the MLP scorer: 0 for sizes outside the contract,
    every n <= 4096 with hidden <= 131072 within the static buffer, and a
    short workspace refused before anything is launched."""
    import ctypes

    from paper_2608_08020_amd import gambit
    L = gambit.lib()
    ws = L.gambit_mlp_workspace_size
    assert ws(0, 64) == 0 and ws(8, 96) == 0 and ws(8, 0) == 0
    assert ws(512, 1024) == 8 * 512 * 1024 * 4       # eight k splits' fp32 partial sums
    assert ws(4096, 16384) == 4096 * (16384 // 128) * 4  # one split: the tiles' partial logits
    assert all(0 < ws(n, hd) <= gambit.MLP_STATIC_SCRATCH_BYTES
               for n in (1, 100, 128, 512, 1000, 4096) for hd in (64, 1024, 4096, 16384, 131072))
    assert ws(4096, 131136) > gambit.MLP_STATIC_SCRATCH_BYTES
    fake = ctypes.c_void_p(1 << 20)              # never dereferenced: the calls fail their checks
    m = gambit.Mlp(256, 128, gambit.ACT_RELU, fake.value, fake.value, fake.value, 0.0)
    need = ws(16, 128)
    assert L.gambit_mlp_score(16, fake, ctypes.byref(m), fake, None, 0, None, fake, need - 1,
                              None) == gambit.ERR_WORKSPACE
