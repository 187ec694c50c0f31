"""Summarise rocprofv3 output of the bench into profiles/ (text only).

    python -m paper_2608_08020_amd.profiling trace --kt DIR/PREFIX ... --out profiles/X.md
    python -m paper_2608_08020_amd.profiling counters --pmc DIR/PREFIX [--pmc ...] ... --out profiles/Y.md

The bench replays its schedule R times, each replay running P attention
launches (the first interval, the warm-up and the timed steps) before the
next starts; the timed steps are launches a .. b (0-based steps) of each
replay.  Both subcommands select exactly those launches of the attention
kernel, in dispatch order, so a summary describes the pool state the bench
line timed.

* trace: a `rocprofv3 --kernel-trace --stats` run of the bench, plus
  `--pmc FETCH_SIZE` / `--pmc WRITE_SIZE` runs of it and of hbm_calib.py (a
  plain copy of known size: counter / true bytes gives the scale applied to
  the attention kernel's counts).  Writes the markdown summary and the
  matching record of profiles/attn_traffic.json (per-launch HBM bytes keyed
  by workload, timed steps and the hash of the attention kernel and planner
  sources; bench.py reports `traffic` only for an exact match).
* counters: `rocprofv3 --pmc ...` runs (one counter set each); every counter
  is averaged over the selected dispatches, and the derived figures
  (occupancy, matrix-core and memory-unit activity, L2 hit rate) are
  computed from them.
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
KERNEL = "attn_units_kernel"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attn_traffic.json")
# the attention kernel's traffic depends on its code, the plan it runs and the cache layout
TRAFFIC_SOURCES = ("decode_attn.hip", "gambit_pool.cpp", "kernels.h")
N_CU, N_XCD, SIMD_PER_CU = 256, 8, 4


def source_sha() -> str:
    h = hashlib.sha256()
    for name in TRAFFIC_SOURCES:
        with open(os.path.join(HERE, "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def _rows(path):
    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def _select(n_total, per_replay, a, b):
    """Indices (in dispatch order) of launches a..b of every replay."""
    if n_total % per_replay:
        raise SystemExit(f"{n_total} attention launches is not a multiple of {per_replay} per replay")
    return [r * per_replay + i for r in range(n_total // per_replay) for i in range(a, b + 1)]


def _dispatch_values(prefix, kernel_sub, counter):
    """Per-dispatch values of one counter, in dispatch order."""
    vals = {}
    for r in _rows(prefix + "_counter_collection.csv"):
        if kernel_sub in r["Kernel_Name"] and r["Counter_Name"] == counter:
            d = int(r["Dispatch_Id"])
            vals[d] = vals.get(d, 0.0) + float(r["Counter_Value"])
    return [vals[d] for d in sorted(vals)]


def _counters_of(prefix, kernel_sub):
    names = sorted({r["Counter_Name"] for r in _rows(prefix + "_counter_collection.csv")
                    if kernel_sub in r["Kernel_Name"]})
    return {n: _dispatch_values(prefix, kernel_sub, n) for n in names}


def _mean_selected(vals, per_replay, a, b):
    idx = _select(len(vals), per_replay, a, b)
    return sum(vals[i] for i in idx) / len(idx), len(idx)


def cmd_trace(a):
    from .hbm_calib import COPY_BYTES

    stats = _rows(a.kt + "_kernel_stats.csv")
    trace = [r for r in _rows(a.kt + "_kernel_trace.csv") if r["Kernel_Name"] == KERNEL]
    trace.sort(key=lambda r: int(r["Start_Timestamp"]))
    durs = [int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in trace]
    sel = _select(len(durs), a.per_replay, a.first, a.last)
    avg_us = sum(durs[i] for i in sel) / len(sel) / 1e3
    per_rep = []
    for r in range(len(durs) // a.per_replay):
        idx = [i for i in sel if i // a.per_replay == r]
        per_rep.append(sum(durs[i] for i in idx) / len(idx) / 1e3)
    cf = sum(_dispatch_values(a.calib_fetch, "copyBuffer", "FETCH_SIZE")) / len(
        _dispatch_values(a.calib_fetch, "copyBuffer", "FETCH_SIZE"))
    cw = sum(_dispatch_values(a.calib_write, "copyBuffer", "WRITE_SIZE")) / len(
        _dispatch_values(a.calib_write, "copyBuffer", "WRITE_SIZE"))
    f_scale = COPY_BYTES / (cf * 1024.0)
    w_scale = COPY_BYTES / (cw * 1024.0)
    fk, nf = _mean_selected(_dispatch_values(a.fetch, KERNEL, "FETCH_SIZE"), a.pmc_per_replay, a.first, a.last)
    wk, nw = _mean_selected(_dispatch_values(a.write, KERNEL, "WRITE_SIZE"), a.pmc_per_replay, a.first, a.last)
    fetch_b = fk * 1024.0 * f_scale
    write_b = wk * 1024.0 * w_scale
    sha = source_sha()
    bench = json.loads(open(a.bench).read().strip().splitlines()[-1]) if a.bench else None
    alg = bench["roofline"]["alg_bytes_per_launch"] if bench else None
    rec = {"workload": a.workload, "timed_steps": [a.first, a.last], "kernel_sha": sha,
           "bytes_per_launch": round(fetch_b + write_b), "fetch_bytes_per_launch": round(fetch_b),
           "write_bytes_per_launch": round(write_b), "fetch_scale": round(f_scale, 4),
           "write_scale": round(w_scale, 4), "dispatches_sampled": min(nf, nw),
           "kernel_trace_avg_us": round(avg_us, 2)}
    try:
        recs = json.load(open(TRAFFIC_FILE))
        recs = recs if isinstance(recs, list) else [recs]
    except (OSError, ValueError):
        recs = []
    recs = [r for r in recs if not (r.get("workload") == a.workload and r.get("timed_steps") == [a.first, a.last])
            and r.get("kernel_sha") == sha]
    recs.append(rec)
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(recs, f, indent=1)
    cmds = open(a.cmds).read().strip()
    lines = [f"# {KERNEL} - {a.workload}, steps {a.first}-{a.last}", "",
             f"The attention launches of decode steps {a.first}-{a.last} of each bench replay (the state the bench "
             f"line times: after the first round and the warm-up), selected in dispatch order "
             f"({a.per_replay} attention launches per replay).", "",
             "Commands (run from the repository root on an MI355X):", "", "```", cmds, "```", "",
             "## Kernel time (rocprofv3 --kernel-trace --stats)", "",
             "| kernel | calls | avg us | total % |", "|---|---|---|---|"]
    for r in stats[:10]:
        lines.append(f"| {r['Name']} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                     f"{float(r['Percentage']):.2f} |")
    lines += ["", f"{KERNEL}, the {len(sel)} timed launches: average **{avg_us:.1f} us** "
              f"(per replay: {', '.join(f'{x:.1f}' for x in per_rep)})"
              + (f"; the bench line's HIP events: {bench['roofline']['avg_launch_us']:.1f} us" if bench else "")
              + ".", ""]
    if alg:
        lines += [f"Algorithmic bytes per launch (bench): {alg / 1e9:.3f} GB -> {alg / avg_us / 1e3:.1f} GB/s "
                  f"= **{alg / avg_us / 1e3 / 8000:.4f}** of 8 TB/s over the kernel-trace average.", ""]
    lines += ["## HBM traffic per launch (rocprofv3 --pmc, one counter per run, one replay)", "",
              f"* copy calibration ({COPY_BYTES >> 20} MiB copy): FETCH_SIZE reads {cf:.0f} KiB, "
              f"WRITE_SIZE {cw:.0f} KiB -> scales {f_scale:.3f} (fetch), {w_scale:.3f} (write)",
              f"* {KERNEL}, the {nf} timed dispatches: FETCH_SIZE {fk:.0f} KiB -> {fetch_b / 1e9:.3f} GB; "
              f"WRITE_SIZE {wk:.0f} KiB -> {write_b / 1e9:.3f} GB",
              f"* total {(fetch_b + write_b) / 1e9:.3f} GB per launch"
              + (f" vs {alg / 1e9:.3f} GB algorithmic ({(fetch_b + write_b) / alg:.3f}x)" if alg else ""),
              f"* sha256[:16] of {' + '.join(TRAFFIC_SOURCES)} = {sha}", ""]
    with open(a.out, "w") as f:
        f.write("\n".join(lines))
    print("\n".join(lines))


def cmd_counters(a):
    vals = {}
    for prefix in a.pmc:
        for name, v in _counters_of(prefix, KERNEL).items():
            vals[name] = _mean_selected(v, a.pmc_per_replay, a.first, a.last)
    g = lambda n: vals[n][0] if n in vals else None  # noqa: E731
    cmds = open(a.cmds).read().strip()
    lines = [f"# {KERNEL} counters - {a.workload}, steps {a.first}-{a.last}", "",
             f"Hardware counters of the attention launches of decode steps {a.first}-{a.last} (the state the bench "
             f"line times), each averaged over those dispatches; one counter set per run (rocprofv3 does not split "
             f"counters over passes).", "",
             "Commands (run from the repository root on an MI355X):", "", "```", cmds, "```", "",
             "| counter | per dispatch | dispatches |", "|---|---|---|"]
    for n in sorted(vals):
        lines.append(f"| {n} | {vals[n][0]:.4g} | {vals[n][1]} |")
    lines += ["", "Derived (GRBM_GUI_ACTIVE sums the 8 XCDs; SQ_WAVE_CYCLES counts in units of 4 cycles; "
              "SQ_VALU_MFMA_BUSY_CYCLES sums the SIMDs):", ""]
    cyc = g("GRBM_GUI_ACTIVE") / N_XCD if g("GRBM_GUI_ACTIVE") else None
    if cyc:
        lines.append(f"* launch length under the counters: {cyc:.4g} cycles per XCD ({cyc / 2.4e3:.1f} us at 2.4 GHz)")
    if cyc and g("SQ_WAVE_CYCLES"):
        occ = 4 * g("SQ_WAVE_CYCLES") / (cyc * N_CU)
        lines.append(f"* occupancy: {occ:.2f} resident waves per CU on average")
    if cyc and g("SQ_VALU_MFMA_BUSY_CYCLES"):
        lines.append(f"* matrix cores busy {g('SQ_VALU_MFMA_BUSY_CYCLES') / (cyc * N_CU * SIMD_PER_CU):.1%} of SIMD "
                     f"cycles")
    if g("SQ_INSTS_VALU_MFMA_BF16") and g("SQ_INSTS_VALU"):
        mf = g("SQ_INSTS_VALU_MFMA_BF16")
        lines.append(f"* {mf:.4g} bf16 MFMA instructions (16x16x32: {mf * 16384 / 1e9:.0f} GFLOP) against "
                     f"{g('SQ_INSTS_VALU'):.4g} VALU instructions ({mf / g('SQ_INSTS_VALU'):.1%} of them MFMA)")
    if g("SQ_WAIT_INST_ANY") and g("SQ_ACTIVE_INST_ANY"):
        lines.append(f"* waves wait {g('SQ_WAIT_INST_ANY') / g('SQ_ACTIVE_INST_ANY'):.2f}x as many cycles as they "
                     f"issue")
    if g("TCC_HIT_sum") is not None and g("TCC_MISS_sum") is not None:
        h, m = g("TCC_HIT_sum"), g("TCC_MISS_sum")
        lines.append(f"* L2 hit rate {h / (h + m):.1%} ({h:.4g} hits, {m:.4g} misses)")
    if g("GRBM_TA_BUSY") is not None and g("GRBM_GUI_ACTIVE"):
        lines.append(f"* memory unit busy (MemUnitBusy; this rocprofv3 has no derived metric of that name): some "
                     f"texture-addresser (TA) unit busy {g('GRBM_TA_BUSY') / g('GRBM_GUI_ACTIVE'):.1%} of the "
                     f"GPU-busy cycles (GRBM_TA_BUSY / GRBM_GUI_ACTIVE)"
                     + (f"; each TA busy {g('TA_BUSY_avr') / cyc:.1%} of the cycles on average (TA_BUSY_avr)"
                        if g("TA_BUSY_avr") is not None and cyc else ""))
    if g("SQ_LDS_BANK_CONFLICT") is not None:
        lines.append(f"* LDS bank conflicts: {g('SQ_LDS_BANK_CONFLICT'):.0f} cycles per launch")
    lines += [f"* sha256[:16] of {' + '.join(TRAFFIC_SOURCES)} = {source_sha()}", ""]
    with open(a.out, "w") as f:
        f.write("\n".join(lines))
    print("\n".join(lines))


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    for name in ("trace", "counters"):
        p = sub.add_parser(name)
        p.add_argument("--workload", required=True)
        p.add_argument("--first", type=int, required=True, help="first timed step")
        p.add_argument("--last", type=int, required=True, help="last timed step")
        p.add_argument("--pmc-per-replay", type=int, required=True,
                       help="attention launches per replay in the counter runs")
        p.add_argument("--out", required=True)
        p.add_argument("--cmds", required=True, help="file with the commands that made the inputs")
        if name == "trace":
            for x in ("kt", "fetch", "write", "calib_fetch", "calib_write"):
                p.add_argument("--" + x.replace("_", "-"), required=True)
            p.add_argument("--per-replay", type=int, required=True, help="attention launches per replay")
            p.add_argument("--bench", default=None, help="the bench's JSON output (last line)")
        else:
            p.add_argument("--pmc", action="append", required=True)
    a = ap.parse_args()
    (cmd_trace if a.cmd == "trace" else cmd_counters)(a)


if __name__ == "__main__":
    main()
