"""The library's host code under sanitizers, on the CPU.

tests/host/mirror_check.cpp compiles the pool's host source (validation,
host mirror, shared-run planner with its host threads, staging copies into
the workspace) with g++ against a host-only HIP stand-in and runs operation
sequences read from stdin.  Built twice - AddressSanitizer + Undefined-
BehaviorSanitizer, and ThreadSanitizer - and driven by random operation
sequences (hypothesis and seeded), it must run clean, and after every
operation its mirror must equal the oracle's pool model (oracle/pool.py):
lengths, block rows, refcounts and free count bit-exact, the same error
for a call the model rejects, and nothing changed by a rejected call.
Every plan a decode step launches must cover each listed trace's context
exactly once per KV head with the blocks its own row lists, use each of the
trace's partial slots exactly once, and report the step's statistics.
"""
from __future__ import annotations

import json
import os
import random
import shutil
import subprocess

import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

from oracle.pool import PoolError, PoolModel

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "host", "mirror_check.cpp")
CODES = {"INVALID": -1, "OUT_OF_BLOCKS": -2, "SHARED_WRITE": -3, "UNSUPPORTED": -4}
SAN = {"asan": ["-fsanitize=address,undefined", "-fno-sanitize-recover=all"], "tsan": ["-fsanitize=thread"]}


def _build(kind, out_dir):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = os.path.join(out_dir, f"mirror_check_{kind}")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", *SAN[kind], "-Wno-subobject-linkage",
           "-I", os.path.join(ROOT, "tests", "host"), "-pthread", SRC, "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    return exe


@pytest.fixture(scope="module")
def harness(tmp_path_factory):
    d = str(tmp_path_factory.mktemp("host_san"))
    return {k: _build(k, d) for k in SAN}


def _run(exe, lines):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", TSAN_OPTIONS="halt_on_error=1:exitcode=66")
    r = subprocess.run([exe], input="\n".join(lines) + "\n", capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0 and "Sanitizer" not in r.stderr and "runtime error" not in r.stderr, \
        f"exit {r.returncode}\n{r.stderr[-6000:]}"
    return [json.loads(x) for x in r.stdout.splitlines()]


# ------------------------------------------------------------- sequences --
def random_ops(rng: random.Random, T: int, n_ops: int, nb: int):
    """A population's life: roots written, forks at unaligned lengths, decode
    steps of subsets (or of everyone), frees, plus invalid calls."""
    ops = []
    live = set()
    for _ in range(n_ops):
        r = rng.random()
        empty = [t for t in range(T) if t not in live]
        if r < 0.18 and empty:
            ts = rng.sample(empty, min(len(empty), rng.randint(1, 3)))
            ops.append(("alloc", [(t, rng.randint(1, 90)) for t in ts]))
            live |= set(ts)
            for t, _ in ops[-1][1]:
                ops.append(("write", (t, 0, 1)))
        elif r < 0.4 and live and empty:
            par = rng.sample(sorted(live), min(len(live), rng.randint(1, 4)))
            ch = rng.sample(empty, min(len(empty), len(par)))
            ops.append(("fork", list(zip(par, ch))))
            live |= set(ch)
        elif r < 0.5 and live:
            ts = rng.sample(sorted(live), min(len(live), rng.randint(1, 3)))
            ops.append(("free", ts))
            live -= set(ts)
        elif r < 0.95 and live:
            ids = sorted(live) if rng.random() < 0.5 else rng.sample(sorted(live), rng.randint(1, len(live)))
            rng.shuffle(ids)
            for _ in range(rng.randint(1, 20)):
                ops.append(("decode", list(ids)))
        else:  # invalid calls: an empty trace, a duplicate, too many tokens
            t = rng.randrange(T)
            choice = rng.randrange(4)
            if choice == 0:
                ops.append(("decode", [t, t]))
            elif choice == 1:
                ops.append(("free", [t] if t not in live else [t, t]))
            elif choice == 2:
                ops.append(("alloc", [(t, nb * 16)]))
            else:
                ops.append(("fork", [(t, t)]))
    return ops


def _line(op):
    kind, arg = op
    if kind in ("alloc", "fork"):
        return kind + " " + " ".join(f"{a} {b}" for a, b in arg)
    if kind == "write":
        return "write {} {} {}".format(*arg)
    return kind + " " + " ".join(str(x) for x in arg)


def _apply_model(m: PoolModel, op, Hkv):
    kind, arg = op
    try:
        if kind == "alloc":
            m.alloc([a for a, _ in arg], [b for _, b in arg])
        elif kind == "write":
            t, p0, n = arg
            z = np.zeros((n, Hkv, 128), np.uint16)
            m.write(t, p0, z, z)
        elif kind == "fork":
            m.fork([a for a, _ in arg], [b for _, b in arg])
        elif kind == "free":
            m.free_traces(arg)
        elif kind == "decode":
            z = np.zeros((len(arg), Hkv, 128), np.uint16)
            if len(set(arg)) != len(arg):
                raise PoolError("INVALID", "duplicate")
            m.append(arg, z, z)
    except PoolError as e:
        return CODES[e.code]
    return 0


def _check_state(st_json, m: PoolModel, where):
    assert st_json["nfree"] == len(m.free), where
    assert st_json["seq_len"] == m.seq_len, where
    assert st_json["refcount"] == m.refcount, where
    assert st_json["rows"] == [list(r) for r in m.table], where


def _check_plan(plan, m: PoolModel, Hkv, g, where):
    ids = plan["list"]
    n = len(ids)
    U = plan["units"]
    mem = plan["members"]
    nk = plan["nk"]
    xo = plan["xcd_off"]
    assert all(xo[i] <= xo[i + 1] and (xo[i + 1] - xo[i]) % 4 == 0 for i in range(8)), where
    assert xo[0] == 0 and xo[8] == len(U), where
    assert plan["grid"] % 8 == 0 and plan["grid"] * 4 >= len(U) - 8 * 4 * 96, where
    assert all(0 < k <= plan["kmax"] for k in nk), where
    cover = {(pos, h): [] for pos in range(n) for h in range(Hkv)}
    for s0 in range(0, len(U), 4):
        slot = U[s0:s0 + 4]
        if slot[0][7] & 1:  # a cooperative item fills the whole slot
            assert all(u == slot[0] for u in slot), where
            slot = slot[:1]
            # up to 128 rows; the last item of a wide chunk takes what is
            # left, as little as one member
            assert 0 < slot[0][5] * g <= 128, where
        for owner, jb0, nblk, kvh, moff, mcnt, kidx, _ in slot:
            if mcnt == 0:
                continue
            assert 0 <= kvh < Hkv, where
            members = mem[moff:moff + mcnt]
            assert members == sorted(members) and len(set(members)) == mcnt, where
            orow = m.table[owner]
            end = len(orow) if nblk < 0 else jb0 + nblk
            assert 0 <= jb0 < end <= len(orow), (where, owner, jb0, nblk)
            for pos in members:
                t = ids[pos]
                assert m.table[t][jb0:end] == orow[jb0:end], (where, "unit reads blocks not in the member's row")
                if nblk < 0:
                    assert t == owner, where
                cover[(pos, kvh)].append((jb0, end, kidx))
    for (pos, h), parts in cover.items():
        t = ids[pos]
        nb = len(m.table[t])
        blocks = sorted((a, b) for a, b, _ in parts)
        at = 0
        for a, b in blocks:
            assert a == at, (where, "trace", t, "head", h, "covered", blocks)
            at = b
        assert at == nb, (where, "trace", t, "head", h, "covered", blocks, "of", nb)
        assert sorted(k for _, _, k in parts) == list(range(nk[pos])), (where, t, h)
    assert all(k != 0 for k in plan["kinds"]), where
    # statistics of the step (after its append)
    used = {b for t in ids for b in m.table[t]}
    total = sum(m.seq_len[t] for t in ids)
    uniq_tok = 16 * len(used) - sum((16 - m.seq_len[t] % 16) % 16 for t in ids)
    assert plan["stats"] == [total, uniq_tok, len(used), sum(len(m.table[t]) for t in ids)], where


def replay_ops(exe, ops, *, nb, Hq, Hkv, T, maxb, splits):
    lines = [f"create {nb} {Hq} {Hkv} {T} {maxb} {splits}", "state"]
    for op in ops:
        lines.append(_line(op))
        lines.append("state")
    out = _run(exe, lines)
    assert out[0]["status"] == 0
    m = PoolModel(num_blocks=nb, n_kv_heads=Hkv, head_dim=128, kv_dtype="bf16", max_traces=T,
                  max_blocks_per_trace=maxb)
    _check_state(out[1], m, "initial")
    k = 2
    plans = 0
    applied = []
    for i, op in enumerate(ops):
        reply, state = out[k], out[k + 1]
        k += 2
        want = _apply_model(m, op, Hkv)
        if reply["status"] == CODES["UNSUPPORTED"] and want == 0:
            # the partial limit (max_splits) is a property of the plan, not of
            # the model: the call must have changed nothing
            m = PoolModel(num_blocks=nb, n_kv_heads=Hkv, head_dim=128, kv_dtype="bf16", max_traces=T,
                          max_blocks_per_trace=maxb)
            for op2 in applied:
                assert _apply_model(m, op2, Hkv) == 0
            _check_state(state, m, f"op {i} {op[0]} (unsupported)")
            continue
        if want == 0:
            applied.append(op)
        assert reply["status"] == want, (i, op, reply["status"], want)
        _check_state(state, m, f"op {i} {op[0]}")
        if op[0] == "decode" and want == 0:
            _check_plan(reply, m, Hkv, Hq // Hkv, f"op {i}")
            plans += 1
    return plans


SHAPES = [(8, 2), (32, 8), (16, 1), (64, 8), (4, 4)]


@settings(max_examples=25, deadline=None, suppress_health_check=[HealthCheck.function_scoped_fixture])
@given(seed=st.integers(0, 2 ** 31 - 1), shape=st.sampled_from(SHAPES), splits=st.sampled_from([0, 4, 64]))
def test_mirror_and_planner_match_the_pool_model_under_asan_ubsan(harness, seed, shape, splits):
    rng = random.Random(seed)
    Hq, Hkv = shape
    T = rng.choice([6, 12, 40])
    nb = rng.choice([40, 120, 400])
    replay_ops(harness["asan"], random_ops(rng, T, 60, nb), nb=nb, Hq=Hq, Hkv=Hkv, T=T, maxb=24, splits=splits)


def test_large_population_under_asan_ubsan(harness):
    """Lists of 130-160 traces: the planner scans rows on host threads."""
    rng = random.Random(1)
    plans = replay_ops(harness["asan"], random_ops(rng, 160, 300, 3000), nb=3000, Hq=32, Hkv=8, T=160, maxb=40,
                       splits=0)
    assert plans > 50


def test_planner_threads_under_tsan(harness):
    """The planner's threaded row scans (lists of 128 or more traces), with
    forks and frees between the steps, under ThreadSanitizer."""
    rng = random.Random(2)
    T = 200
    ops = [("alloc", [(t, rng.randint(20, 200)) for t in range(0, T, 2)])]
    ops.append(("fork", [(t, t + 1) for t in range(0, T, 2)]))
    ids = list(range(T))
    for r in range(6):
        for _ in range(5):
            ops.append(("decode", ids))
        victims = rng.sample(ids, 40)
        ops.append(("free", victims))
        survivors = [t for t in ids if t not in victims]
        ops.append(("fork", list(zip(rng.sample(survivors, 40), victims))))
    plans = replay_ops(harness["tsan"], ops, nb=6000, Hq=32, Hkv=8, T=T, maxb=40, splits=0)
    assert plans == 30
