"""GPU parity of the whole hot path against the oracle, per workload.

Every test drives the C ABI (through the ctypes binding) and compares with
the fp64 oracle on the same seeded inputs; see _parity.py for the bar.
"""
import numpy as np
import pytest
import torch

from _parity import replay
from paper_2608_08020_amd.gambit import UNIT_COOP_ONE, UNIT_COOP_TWO, UNIT_NARROW, UNIT_NARROW_TWO, UNIT_TAIL_SLOT
from workload import CONFIGS, Workload, tiny

KINDS = {UNIT_NARROW: "narrow", UNIT_NARROW_TWO: "narrow, two row blocks", UNIT_COOP_ONE: "cooperative, one row block per wave",
         UNIT_COOP_TWO: "cooperative, two row blocks per wave",
         UNIT_TAIL_SLOT: "slot claimed at run time"}


class PlanCover:
    """Picks, at a sampled step, at least `want` traces that together cover
    every kind of work unit the step's plan uses (a few of each kind, the rest
    at random), and remembers which kinds were covered."""

    def __init__(self, want=32, per_kind=6):
        self.want, self.per_kind, self.seen = want, per_kind, set()

    def __call__(self, run, step):
        kinds = run.pool.plan_kinds(run.ids)
        rng = np.random.default_rng(step)
        chosen = set()
        for bit in KINDS:
            have = np.flatnonzero(kinds & bit)
            if len(have):
                self.seen.add(bit)
                chosen |= set(rng.choice(have, size=min(self.per_kind, len(have)), replace=False).tolist())
        for t in rng.permutation(len(kinds)).tolist():
            if len(chosen) >= self.want:
                break
            chosen.add(t)
        return sorted(chosen)

pytestmark = pytest.mark.gpu


def test_tiny_bf16_every_step_every_trace():
    replay(Workload(tiny()), check_pool_every_step=True)


def test_tiny_bf16_output_dtype_bf16():
    replay(Workload(tiny()), out_dtype=torch.bfloat16)


def test_tiny_fp8_every_step_every_trace():
    replay(Workload(tiny("fp8_e4m3")), check_pool_every_step=True)


def test_tiny_wide_group_many_row_tiles():
    # 48 traces x g = 8 share the prompt: 384 rows, three 128-row tiles
    cfg = tiny(n_q_heads=16, n_kv_heads=2, gens=(3, 12, 48), keep=12, n_parents=12, steps=20)
    replay(Workload(cfg), sample_steps=[0, 15, 16, 19])


def test_cfg1_8_traces():
    replay(Workload(CONFIGS[1]))


def test_cfg2_64_traces():
    wl = Workload(CONFIGS[2])
    steps = sorted({0, 1, 255} | {s for r in wl.rounds_after() for s in (r, r + 1) if s < 256})
    replay(wl, sample_steps=steps)


@pytest.mark.timeout(900)
def test_cfg3_256_traces_sampled():
    wl = Workload(CONFIGS[3])
    steps = sorted({0, 511} | {r + 1 for r in wl.rounds_after() if r + 1 < 512})
    replay(wl, sample_steps=steps, sample_traces=[0, 1, 63, 64, 130, 191, 200, 255])


@pytest.mark.timeout(900)
def test_cfg5_fp8_256_traces_sampled():
    wl = Workload(CONFIGS[5])
    steps = sorted({0, 511} | {r + 1 for r in wl.rounds_after() if r + 1 < 512})
    replay(wl, sample_steps=steps, sample_traces=[0, 5, 64, 99, 128, 200, 255])


@pytest.mark.timeout(900)
def test_cfg5_fp8_quantise_on_append_sampled():
    """The fp8 workload with bf16 new K/V quantised by the pool on append
    (landing block's scale; decode-opened blocks at the append scale) across
    the first round."""
    wl = Workload(CONFIGS[5], total_steps=140)
    replay(wl, sample_steps=[0, 15, 16, 127, 128, 139], sample_traces=[0, 5, 64, 99, 200, 255],
           quantise_on_append=True)


@pytest.mark.timeout(1200)
def test_cfg4_512_traces_full_size_sampled():
    """The benchmarked workload at full size, in the bench's launch configuration."""
    wl = Workload(CONFIGS[4])
    steps = [0, 256, 1023]
    replay(wl, sample_steps=steps, sample_traces=[0, 129, 300, 511], share_nodes=False,
           out_dtype=torch.bfloat16)


@pytest.mark.timeout(1200)
def test_cfg4_512_traces_full_size_fp32_strict():
    """The benchmarked workload at full size and fp32 output, at the plain
    elementwise bar 1e-3 + 2e-3 |ref|: at the first step, the first step after
    each of the three rounds and the last, 32+ traces chosen from that step's
    plan so that every kind of work unit is checked (narrow units, cooperative
    items with one and with two row blocks per wave, slots claimed at run
    time)."""
    wl = Workload(CONFIGS[4])
    cover = PlanCover(want=32)
    steps = sorted({0, wl.total_steps - 1} | {r + 1 for r in wl.rounds_after() if r + 1 < wl.total_steps})
    assert steps == [0, 256, 512, 768, 1023]
    replay(wl, sample_steps=steps, sample_traces=cover, share_nodes=False, out_dtype=torch.float32)
    want = {UNIT_NARROW, UNIT_COOP_ONE, UNIT_COOP_TWO, UNIT_TAIL_SLOT}
    assert want <= cover.seen, f"kinds not covered: {[KINDS[k] for k in want - cover.seen]}"


@pytest.mark.timeout(900)
def test_cfg5_fp8_covers_every_unit_kind():
    """The fp8 workload's chunks of 17-32 rows run as narrow units of two row
    blocks; traces chosen from the plan so that those units, one-block narrow
    units and cooperative items are all checked, before and after the first
    round."""
    wl = Workload(CONFIGS[5], total_steps=140)
    cover = PlanCover(want=24)
    replay(wl, sample_steps=[0, 129, 139], sample_traces=cover)
    want = {UNIT_NARROW, UNIT_NARROW_TWO, UNIT_COOP_ONE}
    assert want <= cover.seen, f"kinds not covered: {[KINDS[k] for k in want - cover.seen]}"
