"""The tournament workloads, run on the oracle alone (CPU): the events they
schedule make every part of Alg. 1's loop happen - both tournament cases,
evictions into ghosts, ghosts pruned, completions - with no near-tie at any
ranking decision (the driver asserts that), so the GPU comparison of the same
run is exact; and the counts are conserved (App. A.5's identity)."""
import pytest

from _tournament import run
from workload.tournament import TOURNAMENT_SMALL


def test_small_run_exercises_the_whole_loop():
    st = run(TOURNAMENT_SMALL, use_gpu=False)
    assert st["case1"] > 0 and st["case2"] > 0
    assert st["evictions"] > 0 and st["ghosts_pruned"] > 0 and st["completions"] > 0
    assert st["alive"] == TOURNAMENT_SMALL.roots + st["branches"] - st["prunes"] - st["completions"]
