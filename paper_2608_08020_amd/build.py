"""Build libgambit.so for gfx950 in-tree with hipcc.

    python -m paper_2608_08020_amd.build

The library holds the host mirror/planner (C++17) and the HIP kernels.  All
device code is compiled with packed-fp32 instructions disabled.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libgambit.so")
SOURCES = ["gambit_pool.cpp", "blocktable.hip", "decode_attn.hip", "probe_topk.hip", "mlp_scorer.hip",
           "seq_scorer.cpp", "seqscorer.hip", "membench.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall", "-mcode-object-version=5",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include"), "-I", CSRC]


# The attention kernel takes maxima of matrix-core results.  In IEEE mode
# every such max first quiets its operands (one extra instruction each); no
# NaN ever reaches a max there (cache slots past a chunk's end are replaced
# by a select before any max), so that source is built without IEEE mode.
EXTRA = {"decode_attn.hip": ["-fno-honor-nans", "-mno-amdgpu-ieee"]}


def build(verbose: bool = False) -> str:
    build_dir = os.path.join(HERE, "_build")
    os.makedirs(build_dir, exist_ok=True)

    def compile_one(src):
        obj = os.path.join(build_dir, src + ".o")
        cmd = [HIPCC, *FLAGS, *EXTRA.get(src, []), "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed on {src}:\n{r.stderr}")
        return obj

    jobs = max(1, min(len(SOURCES), len(os.sched_getaffinity(0)), 8))
    with ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-pthread", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
