"""Summarise rocprofv3 output of the bench into profiles/ (text only).

    python -m paper_2608_08020_amd.profiling \
        --kt DIR/PREFIX --fetch DIR/PREFIX --write DIR/PREFIX \
        --calib-fetch DIR/PREFIX --calib-write DIR/PREFIX \
        --workload NAME --timed K --sampled S --out profiles/NAME.md --cmds FILE

* --kt: a `rocprofv3 --kernel-trace --stats` run of bench.py; the kernel's
  average duration is taken over its last K launches (the timed steps).
* --fetch / --write: `rocprofv3 --pmc FETCH_SIZE` / `--pmc WRITE_SIZE` runs;
  the last S attention dispatches are averaged.
* --calib-*: the same counters over hbm_calib.py, a plain copy of known
  size; counter / true bytes gives the scale applied to the attention counts.
Writes the markdown summary and profiles/attn_traffic.json (per-launch HBM
bytes keyed by the hash of the attention kernel and planner sources, which
bench.py reports only while both are unchanged).
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
# the attention kernel's traffic depends on its code and on the plan it runs
TRAFFIC_SOURCES = ("decode_attn.hip", "gambit_pool.cpp")


def source_sha() -> str:
    h = hashlib.sha256()
    for name in TRAFFIC_SOURCES:
        with open(os.path.join(HERE, "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def _rows(path):
    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def _counter(prefix, kernel_sub, counter, last=None):
    rows = [r for r in _rows(prefix + "_counter_collection.csv")
            if kernel_sub in r["Kernel_Name"] and r["Counter_Name"] == counter]
    vals = [float(r["Counter_Value"]) for r in rows]
    if last:
        vals = vals[-last:]
    return sum(vals) / len(vals), len(vals)


def main():
    ap = argparse.ArgumentParser()
    for a in ("kt", "fetch", "write", "calib_fetch", "calib_write", "workload", "out", "cmds"):
        ap.add_argument("--" + a.replace("_", "-"), required=True)
    ap.add_argument("--timed", type=int, required=True)
    ap.add_argument("--sampled", type=int, required=True)
    ap.add_argument("--alg-bytes", type=float, default=None, help="bench alg_bytes_per_launch")
    ap.add_argument("--bench-us", type=float, default=None, help="bench avg_launch_us")
    a = ap.parse_args()

    from .hbm_calib import COPY_BYTES

    stats = _rows(a.kt + "_kernel_stats.csv")
    trace = [r for r in _rows(a.kt + "_kernel_trace.csv") if r["Kernel_Name"] == KERNEL]
    durs = [int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in trace][-a.timed:]
    avg_us = sum(durs) / len(durs) / 1e3
    cf, _ = _counter(a.calib_fetch, "copyBuffer", "FETCH_SIZE")
    cw, _ = _counter(a.calib_write, "copyBuffer", "WRITE_SIZE")
    f_scale = COPY_BYTES / (cf * 1024.0)
    w_scale = COPY_BYTES / (cw * 1024.0)
    fk, nf = _counter(a.fetch, KERNEL, "FETCH_SIZE", a.sampled)
    wk, nw = _counter(a.write, KERNEL, "WRITE_SIZE", a.sampled)
    fetch_b = fk * 1024.0 * f_scale
    write_b = wk * 1024.0 * w_scale
    sha = source_sha()
    rec = {"workload": a.workload, "kernel_sha": sha, "bytes_per_launch": round(fetch_b + write_b),
           "fetch_bytes_per_launch": round(fetch_b), "write_bytes_per_launch": round(write_b),
           "fetch_scale": round(f_scale, 4), "write_scale": round(w_scale, 4),
           "dispatches_sampled": min(nf, nw)}
    with open(os.path.join(ROOT, "profiles", "attn_traffic.json"), "w") as f:
        json.dump(rec, f, indent=1)
    cmds = open(a.cmds).read().strip()
    lines = [f"# {KERNEL} - {a.workload}", "",
             "Commands (run from the repository root on an MI355X):", "", "```", cmds, "```", "",
             f"## Kernel time (rocprofv3 --kernel-trace --stats)", "",
             "| kernel | calls | avg us | total % |", "|---|---|---|---|"]
    for r in stats[:10]:
        lines.append(f"| {r['Name']} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                     f"{float(r['Percentage']):.2f} |")
    lines += ["", f"{KERNEL}: average over the last {len(durs)} launches (the timed steps) "
              f"= **{avg_us:.1f} us**" + (f"; bench.py's HIP events measured {a.bench_us:.1f} us"
                                          if a.bench_us else "") + ".", "",
              "## HBM traffic per launch (rocprofv3 --pmc, one counter per run)", "",
              f"* copy calibration ({COPY_BYTES >> 20} MiB copy): FETCH_SIZE reads {cf:.0f} KiB, "
              f"WRITE_SIZE {cw:.0f} KiB -> scales {f_scale:.3f} (fetch), {w_scale:.3f} (write)",
              f"* {KERNEL}, last {nf} dispatches: FETCH_SIZE {fk:.0f} KiB -> {fetch_b / 1e9:.3f} GB; "
              f"WRITE_SIZE {wk:.0f} KiB -> {write_b / 1e9:.3f} GB",
              f"* total {(fetch_b + write_b) / 1e9:.3f} GB per launch"
              + (f" vs {a.alg_bytes / 1e9:.3f} GB algorithmic ({(fetch_b + write_b) / a.alg_bytes:.2f}x)"
                 if a.alg_bytes else ""),
              f"* sha256[:16] of {' + '.join(TRAFFIC_SOURCES)} = {sha}", ""]
    with open(a.out, "w") as f:
        f.write("\n".join(lines))
    print("\n".join(lines))


if __name__ == "__main__":
    main()
