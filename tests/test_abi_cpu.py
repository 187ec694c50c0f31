"""The C-ABI library loads on a machine without a GPU and exports every
entry point include/gambit.h declares; host-only queries work."""
import ctypes
import os
import re

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
    for field, bad in [("d_model", 200), ("n_heads", 3), ("input_dim", 100), ("d_ff", 100), ("max_steps", 0),
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
