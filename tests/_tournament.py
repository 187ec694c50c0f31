"""Lock-step driver of a tournament run: the GPU path (through the C ABI)
and the oracle follow the same workload events and are compared every
thought boundary.  The loop follows Alg. 1: Generate (a decode step; at a
thought boundary every running trace completes a thought and is scored),
Schedule (an eviction when the workload says memory is short), Tournament
(at a thought boundary), then completed traces leave.

Bars: thought scores and running means within 1e-5 (fp32 arithmetic against
fp64); eviction victims, tournament cases, pruned ids, (child, parent)
pairs, the ranked tree view, block tables, lengths, GenLen, thought counts
and ghost flags bit-exact; attention as in _parity.ATTN_* .  Exactness of a
ranking decision needs the oracle's scores to be at least GAP apart where
they decide it; the driver asserts that for every decision it meets.
"""
from __future__ import annotations

import math

import numpy as np
import torch

from oracle.attention import decode_attention
from oracle.formats import bf16_to_f64
from oracle.pool import PoolModel
from oracle.probe import probe_scores
from oracle.tournament import TournamentModel
from paper_2608_08020_amd.gambit import Pool
from workload.tournament import TournamentWorkload

GAP = 1e-5
SCORE_TOL = 1e-5


def _bf16_dev(bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def _min_gap(model: TournamentModel, ranked: list, cuts) -> float:
    """Smallest score gap across the given cut positions of the ranking."""
    g = math.inf
    for k in cuts:
        if 0 < k < len(ranked):
            g = min(g, model.sbar[ranked[k - 1]] - model.sbar[ranked[k]])
    return g


def same_ranking(got: list, want: list, sbar: list) -> bool:
    """Equal, except possibly inside runs of scores closer than GAP."""
    if sorted(got) != sorted(want):
        return False
    i = 0
    while i < len(want):
        j = i + 1
        while j < len(want) and sbar[want[j - 1]] - sbar[want[j]] < GAP:
            j += 1
        if set(got[i:j]) != set(want[i:j]):
            return False
        i = j
    return True


def run(cfg, attn_steps=(), sample=3, use_gpu=True):
    """Runs the workload; without the GPU only the oracle side (for CPU checks of the workload)."""
    wl = TournamentWorkload(cfg)
    gpu = Pool(num_blocks=cfg.num_blocks, num_q_heads=cfg.n_q_heads, num_kv_heads=cfg.n_kv_heads,
               max_traces=cfg.slots, max_blocks_per_trace=cfg.max_blocks_per_trace) if use_gpu else None
    om = TournamentModel(PoolModel(num_blocks=cfg.num_blocks, n_kv_heads=cfg.n_kv_heads, head_dim=cfg.head_dim,
                                   kv_dtype="bf16", max_traces=cfg.slots,
                                   max_blocks_per_trace=cfg.max_blocks_per_trace))
    w, b = wl.probe_weights()
    wd = torch.from_numpy(w).cuda() if use_gpu else None
    scale = 1.0 / math.sqrt(cfg.head_dim)
    stats = {"case1": 0, "case2": 0, "evictions": 0, "completions": 0, "ghosts_pruned": 0, "attn_checked": 0,
             "worst_attn": 0.0, "worst_score": 0.0}
    for r, L in enumerate(wl.prompt_lengths()):
        k, v = wl.prompt_kv(r, L)
        if use_gpu:
            gpu.kv_alloc([r], [L])
            gpu.kv_write(r, 0, _bf16_dev(k), _bf16_dev(v))
        om.pool.alloc([r], [L])
        om.pool.write(r, 0, k, v)
    rnd = 0
    for s in range(cfg.steps):
        running = om.scheduler_view()
        if not running:
            break
        # Generate: one decode step for every running trace
        q = wl.step_q(s, len(running))
        kn, vn = wl.step_kv(s, len(running))
        if use_gpu:
            out = gpu.decode_attn(running, _bf16_dev(q), _bf16_dev(kn), _bf16_dev(vn), out_dtype=torch.float32)
        om.pool.append(running, kn, vn)
        om.decoded(running)
        if use_gpu and s in attn_steps:
            o = out.cpu().numpy()
            for i in np.linspace(0, len(running) - 1, min(sample, len(running))).astype(int):
                t = running[i]
                K, V = om.pool.materialise(t)
                ref = decode_attention(bf16_to_f64(q[i]), K, V, scale)
                err = np.abs(o[i] - ref)
                assert (err <= 1e-3 + 2e-3 * np.abs(ref)).all(), f"attention step {s} trace {t}"
                stats["worst_attn"] = max(stats["worst_attn"], float(err.max()))
                stats["attn_checked"] += 1
        boundary = wl.is_boundary(s)
        if boundary:  # every running trace completed a thought
            h = wl.round_h(rnd, len(running))
            f_ref = probe_scores(bf16_to_f64(h), w, b)
            if use_gpu:
                f_gpu = gpu.score_update(running, _bf16_dev(h), wd, b).cpu().numpy()
                err = float(np.abs(f_gpu - f_ref).max())
                assert err <= SCORE_TOL, f"thought scores step {s}: {err}"
                stats["worst_score"] = max(stats["worst_score"], err)
            om.score_update(running, f_ref)
        # Schedule: memory pressure evicts the running trace of lowest running score
        if wl.evicts_at(s) and len(running) > 1:
            ranked = om.rank(running)
            assert _min_gap(om, ranked, [len(ranked) - 1]) >= GAP, f"eviction near-tie at step {s}"
            v_ref = om.evict(running)
            if use_gpu:
                v_gpu = gpu.evict(running)
                assert v_gpu == v_ref, (s, v_gpu, v_ref)
            stats["evictions"] += 1
        # Tournament
        if boundary:
            act = om.tree_view()
            ranked = om.rank(act)
            ghosts_before = {t for t in act if om.ghost[t]}
            n = len(act)
            elig = [t for t in ranked if om.eligible(t, cfg.warmup)]
            if n >= cfg.capacity:
                cut_prune = n - min(cfg.swap_k, n)
                gone = set(ranked[cut_prune:])
                elig = [t for t in elig if t not in gone]
                cuts = [cut_prune]
            else:
                cuts = []
            m = min(cfg.swap_k if n >= cfg.capacity else cfg.capacity - n, len(elig))
            g = _min_gap(om, ranked, cuts)
            if 0 < m < len(elig):
                g = min(g, om.sbar[elig[m - 1]] - om.sbar[elig[m]])
            assert g >= GAP, f"ranking near-tie at step {s}: {g}"
            sbar_before = list(om.sbar)
            res = om.tournament(cfg.capacity, cfg.swap_k, cfg.warmup)
            if use_gpu:
                case, N, pruned, pairs, rk = gpu.tournament(cfg.capacity, cfg.swap_k, cfg.warmup, want_ranked=True)
                assert (case, N) == (res.case, res.n_active), (s, case, N, res.case, res.n_active)
                assert same_ranking(rk, res.ranked, sbar_before), f"ranking step {s}"
                assert pruned == res.pruned, (s, pruned, res.pruned)
                assert pairs == res.pairs, (s, pairs, res.pairs)
            stats[f"case{res.case}"] += 1
            stats["ghosts_pruned"] += len(ghosts_before & set(res.pruned))
            rnd += 1
        # completed traces leave both views
        c = wl.completion_at(s, om.scheduler_view())
        if c is not None:
            if use_gpu:
                gpu.kv_free([c])
            om.complete([c])
            stats["completions"] += 1
        if use_gpu and boundary:
            compare_state(gpu, om, cfg.slots, s)
        om.pool.check_invariants()
    if use_gpu:
        compare_state(gpu, om, cfg.slots, cfg.steps)
    stats["branches"], stats["prunes"] = om.branches, om.prunes
    stats["alive"] = len(om.tree_view())
    return stats


def compare_state(gpu: Pool, om: TournamentModel, T: int, s: int):
    ids = list(range(T))
    sb, ns, ge, gh = gpu.trace_state(ids)
    assert np.abs(sb.astype(np.float64) - np.array(om.sbar)).max() <= SCORE_TOL, f"running means step {s}"
    assert ns.tolist() == om.nsc, f"thought counts step {s}"
    assert ge.tolist() == om.gen, f"GenLen step {s}"
    assert [bool(x) for x in gh] == om.ghost, f"ghost flags step {s}"
    assert gpu.seq_len.cpu().numpy().tolist() == om.pool.seq_len, f"lengths step {s}"
    tab = gpu.block_table.cpu().numpy()
    assert np.array_equal(tab, om.pool.table_array()), f"block tables step {s}"
    assert gpu.refcount.cpu().numpy().tolist() == om.pool.refcount, f"refcounts step {s}"
    gpu.pool_check()
