"""GPU parity of the whole hot path against the oracle, per workload.

Every test drives the C ABI (through the ctypes binding) and compares with
the fp64 oracle on the same seeded inputs; see _parity.py for the bar.
"""
import pytest
import torch

from _parity import replay
from workload import CONFIGS, Workload, tiny

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
