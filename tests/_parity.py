"""Side-by-side replay of a workload on the GPU (through the C ABI) and in the
oracle, with the parity bar:

* attention outputs: |gpu - ref| <= 1e-3 + 2e-3 |ref| elementwise for fp32
  output; a bf16 output additionally carries its own rounding (<= 2^-8 |ref|);
* probe scores: |gpu - ref| <= 1e-4;
* kept ids (in rank order), child -> parent pairs, block tables, lengths and
  refcounts: bit-exact.  Where the oracle's fp64 scores put two traces
  within 1e-6 of each other at a place that decides the selection, either
  order is correct; the GPU's choice is then checked for validity and the
  oracle continues from it.
"""
from __future__ import annotations

import os
import time

import numpy as np
import torch

from oracle import run as orun
from oracle.probe import rank
from workload.generate import to_bf16_bits

ATOL, RTOL = 1e-3, 2e-3
BF16_OUT_REL = 2.0 ** -8
SCORE_TOL = 1e-4
NEAR_TIE = 1e-6

# worst attention error of each replay, by test (printed in pytest's summary)
WORST: dict = {}


def say(msg):
    print(f"[parity] {msg}", flush=True)


def assert_attn_close(gpu: np.ndarray, ref: np.ndarray, what: str, bf16_out: bool = False):
    tol = ATOL + (RTOL + (BF16_OUT_REL if bf16_out else 0.0)) * np.abs(ref)
    err = np.abs(gpu.astype(np.float64) - ref)
    bad = err > tol
    if bad.any():
        i = np.unravel_index(np.argmax(err - tol), err.shape)
        raise AssertionError(f"{what}: {bad.sum()} of {bad.size} outside tolerance; worst at {i}: "
                             f"gpu {gpu[i]!r} ref {ref[i]!r}")
    return float(err.max())


def check_keep(gpu_keep, ids, ref_scores, keep):
    """Returns the keep list the oracle should continue with."""
    ref_keep = rank(ids, ref_scores)[:keep]
    if list(gpu_keep) == ref_keep:
        return ref_keep, False
    sc = {t: float(s) for t, s in zip(ids, ref_scores)}
    g = list(gpu_keep)
    assert len(set(g)) == keep and set(g) <= set(ids), "GPU keep list is not a valid selection"
    for a, b in zip(g, g[1:]):
        assert sc[a] >= sc[b] - NEAR_TIE, f"GPU rank order {a} before {b} is not a near tie"
    worst_kept = min(sc[t] for t in g)
    for t in set(ids) - set(g):
        assert sc[t] <= worst_kept + NEAR_TIE, f"trace {t} pruned although clearly above the cut"
    say(f"near tie resolved by the GPU: {ref_keep} vs {g}")
    return g, True


def compare_tables(run, model, what):
    T = run.T
    tab = run.pool.block_table.cpu().numpy()
    ref = model.table_array(range(T))
    assert np.array_equal(tab[:, :ref.shape[1]], ref), f"{what}: block tables differ"
    assert (run.pool.seq_len.cpu().numpy() == np.array(model.seq_len[:T])).all(), f"{what}: lengths differ"
    rc = run.pool.refcount.cpu().numpy()
    assert (rc == np.array(model.refcount)).all(), f"{what}: refcounts differ"


def replay(wl, *, sample_steps=None, sample_traces=None, out_dtype=torch.float32, num_blocks=None,
           share_nodes=True, check_pool_every_step=False, max_splits=0, quantise_on_append=False):
    """quantise_on_append: the steps' new K/V go in as bf16 and the fp8 pool
    quantises them (the oracle with its own encoder and the landing blocks'
    scales) instead of arriving as the generator's codes.

    sample_traces: list positions to compare at the sampled steps (default
    all), or a callable (run, step) -> positions, called after the step's
    decode (so it can read the plan that step used)."""
    from paper_2608_08020_amd.runner import PopulationRun, estimate_blocks

    t0 = time.time()
    nb = num_blocks or estimate_blocks(wl)
    cache = {}

    def node_data(nid):
        if nid not in cache:
            cache[nid] = wl.node_kv(nid)
        return cache[nid]

    say(f"{wl.cfg.name}: T={wl.T} steps={wl.total_steps} blocks={nb}")
    run = PopulationRun(wl, num_blocks=nb, max_splits=max_splits)
    run.setup(node_data if share_nodes else None)
    model = orun.new_pool(wl, nb)
    if share_nodes:
        for op in wl.setup_ops():
            if op[0] == "fork":
                model.fork(op[1], op[2])
            elif op[0] == "alloc":
                model.alloc(op[1], op[2])
            else:
                k, v, sc = node_data(op[3])
                model.write(op[1], op[2], k, v, sc)
    else:
        orun.apply_setup(model, wl, lazy=True)
        cache.clear()
    run.pool.pool_check()
    compare_tables(run, model, "after setup")
    say(f"setup parity ok ({time.time() - t0:.1f}s)")

    steps = range(wl.total_steps)
    sample_steps = set(steps) if sample_steps is None else set(sample_steps)
    pick = sample_traces if callable(sample_traces) else None
    traces = list(range(wl.T)) if sample_traces is None else (None if pick else list(sample_traces))
    n_checked = 0
    rounds = {s: i for i, s in enumerate(wl.rounds_after())}
    run.load_rounds(range(len(rounds)))
    ids = list(range(wl.T))
    worst = 0.0
    near_ties = 0
    for c0 in range(0, wl.total_steps, 128):
        chunk = list(range(c0, min(wl.total_steps, c0 + 128)))
        run.load_steps(chunk, keep_host=True)
        for s in chunk:
            q, k, v = run.host[s]
            if quantise_on_append:
                x = to_bf16_bits(wl.step_kv_f32(s))
                dev = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()  # noqa: E731
                out = run.pool.decode_attn_layer(0, run.ids, run.q[s], dev(x[0]), dev(x[1]), new_dtype="bf16",
                                                 out_dtype=out_dtype)
                model.append_quantised(ids, x[0], x[1])
            else:
                out = run.decode(s, out_dtype=out_dtype)
                model.append(ids, k, v)
            if s in sample_steps:
                tr = list(pick(run, s)) if pick else traces
                got = out[tr].float().cpu().numpy()
                ref = orun.attend(model, wl, q, tr)
                for i, t in enumerate(tr):
                    worst = max(worst, assert_attn_close(got[i], ref[t], f"step {s} trace {t}",
                                                         bf16_out=out_dtype == torch.bfloat16))
                n_checked += len(tr)
            if check_pool_every_step:
                run.pool.pool_check()
            if s in rounds:
                r = rounds[s]
                scores, keep, pairs = run.round(r)
                h = wl.round_h(r)
                w, b = wl.probe_weights()
                from oracle.formats import bf16_to_f64
                from oracle.probe import probe_scores
                ref_scores = probe_scores(bf16_to_f64(h[ids]), w, b)
                gs = scores.cpu().numpy().astype(np.float64)
                assert np.abs(gs - ref_scores).max() <= SCORE_TOL, f"round {r}: probe scores"
                gk = keep.cpu().numpy().tolist()
                cont, tie = check_keep(gk, ids, ref_scores, wl.cfg.keep)
                near_ties += tie
                _, okeep, opairs = orun.run_round(model, wl, r, ids, keep_override=cont)
                assert gk == okeep
                assert pairs.cpu().numpy().tolist() == [list(p) for p in opairs], f"round {r}: pairs"
                run.pool.pool_check()
                compare_tables(run, model, f"round {r}")
                say(f"round {r} after step {s}: keep/pairs/tables bit-exact")
            del run.host[s], run.q[s], run.kv[s]
    say(f"done: worst |err| {worst:.3g} over {n_checked} (trace, step) outputs, near ties {near_ties}, "
        f"{time.time() - t0:.1f}s")
    test = os.environ.get("PYTEST_CURRENT_TEST", wl.cfg.name).split(" ")[0]
    WORST[test] = (worst, n_checked, "bf16" if out_dtype == torch.bfloat16 else "fp32")
    return run, model, worst
