"""The sequence scorer's incremental inference (App. A.1, Eqs. 4-6) through
the C ABI against the oracle's whole-history forward.

Bar: scores within 1e-5 absolute.  The GPU path is fp32 (weights,
activations, cached keys and values); the oracle fp64.  fp32's unit
roundoff is 6e-8; the longest dot product is 4096 terms (the input
projection), so a logit's relative error stays near 1e-6, and the sigmoid's
slope is at most 1/4.  Step counts bit-exact with the host mirror and the
oracle's histories.
"""
import numpy as np
import pytest
import torch

from oracle.formats import bf16_to_f64
from oracle.seqscorer import SeqScorerModel, scorer_outputs
from paper_2608_08020_amd.gambit import GambitError, Scorer
from workload.seqscorer import SEQ_512, SEQ_SMALL, step_states, weights

pytestmark = pytest.mark.gpu
TOL = 1e-5


def _bf16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def _make(cfg):
    w = weights(cfg)
    gpu = Scorer(w, n_heads=cfg.n_heads, max_steps=cfg.max_steps, max_traces=cfg.slots)
    ref = SeqScorerModel(w, cfg.n_heads, cfg.slots, cfg.max_steps)
    return w, gpu, ref


def test_small_every_round_with_forks_and_frees():
    cfg = SEQ_SMALL
    _, gpu, ref = _make(cfg)
    rng = np.random.default_rng(51)
    live = list(range(10))
    worst = 0.0
    for r in range(36):
        ids = [int(t) for t in rng.permutation(live)[:max(1, int(len(live) * rng.uniform(0.5, 1.0)))]]
        ids = [t for t in ids if ref.hist[t].__len__() < cfg.max_steps]
        H = step_states(cfg, r)[ids]
        got = gpu.step(ids, _bf16(H)).cpu().numpy()
        want = ref.step(ids, bf16_to_f64(H))
        err = float(np.abs(got - want).max())
        worst = max(worst, err)
        assert err <= TOL, (r, err)
        if r % 5 == 4:  # prune two, branch two children from the survivors, into free slots
            gone = [int(t) for t in rng.choice(live, 2, replace=False)]
            gpu.free(gone)
            ref.free(gone)
            live = [t for t in live if t not in gone]
            free_slots = [t for t in range(cfg.slots) if t not in live][:3]
            parents = [int(t) for t in rng.choice(live, len(free_slots))]
            gpu.fork(parents, free_slots)
            ref.fork(parents, free_slots)
            live += free_slots
        assert [gpu.steps(t) for t in range(cfg.slots)] == [len(h) for h in ref.hist]
    gpu.check()
    assert worst > 0  # fp32 against fp64: not bitwise equal, within the bar


def test_full_size_512_traces_sampled():
    cfg = SEQ_512
    w, gpu, _ = _make(cfg)
    ids = np.arange(cfg.slots)
    hist = []
    sample = [0, 77, 255, 256, 511]
    for r in range(24):
        H = step_states(cfg, r)
        hist.append(H)
        got = gpu.step(ids, _bf16(H)).cpu().numpy()
        if r in (0, 1, 7, 23):
            for t in sample:
                Ht = np.stack([bf16_to_f64(h[t]) for h in hist])
                want = scorer_outputs(w, Ht, cfg.n_heads)[-1]
                assert abs(got[t] - want) <= TOL, (r, t, got[t], want)
    # a ragged subset (77 rows: two full 64-row tiles would be 128), then one row
    sub = np.arange(3, 3 + 77)
    H = step_states(cfg, 24)
    got = gpu.step(sub, _bf16(H[sub])).cpu().numpy()
    for i in (0, 40, 76):
        t = int(sub[i])
        Ht = np.stack([bf16_to_f64(h[t]) for h in hist] + [bf16_to_f64(H[t])])
        assert abs(got[i] - scorer_outputs(w, Ht, cfg.n_heads)[-1]) <= TOL
    got1 = gpu.step([511], _bf16(H[511:512])).cpu().numpy()
    Ht = np.stack([bf16_to_f64(h[511]) for h in hist] + [bf16_to_f64(H[511])])
    assert abs(got1[0] - scorer_outputs(w, Ht, cfg.n_heads)[-1]) <= TOL
    assert gpu.steps(0) == 24 and gpu.steps(3) == 25 and gpu.steps(511) == 25
    gpu.check()


def test_errors_change_nothing():
    cfg = SEQ_SMALL
    _, gpu, ref = _make(cfg)
    H = step_states(cfg, 0)
    gpu.step([0, 1], _bf16(H[:2]))
    for bad in ([0, 0], [cfg.slots], [-1]):
        with pytest.raises(GambitError):
            gpu.step(bad, _bf16(H[:len(bad)]))
    with pytest.raises(GambitError):
        gpu.fork([0], [0])
    with pytest.raises(GambitError):
        gpu.fork([2, 1], [1, 3])            # 1 is both child and parent
    for r in range(cfg.max_steps - 1):      # fill slot 0 to its capacity
        gpu.step([0], _bf16(step_states(cfg, r + 1)[:1]))
    assert gpu.steps(0) == cfg.max_steps
    with pytest.raises(GambitError):
        gpu.step([0], _bf16(H[:1]))
    assert gpu.steps(0) == cfg.max_steps and gpu.steps(1) == 1
    gpu.free([0])
    assert gpu.steps(0) == 0
    gpu.check()
    # a freed slot starts a fresh history
    got = gpu.step([0], _bf16(H[5:6])).cpu().numpy()[0]
    assert abs(got - ref.step([0], bf16_to_f64(H[5:6]))[0]) <= TOL


def test_offset_step_states_and_one_input_chunk():
    """Step states with a large common offset (mean 4, spread 0.5: the input
    LayerNorm removes most of each state) and an input width of 128 (one
    k chunk, one split), against the oracle, which normalises first; the
    input LayerNorm's gains are drawn wide (0.1 to 3) and its biases large."""
    import dataclasses
    from workload.generate import to_bf16_bits
    cfg = dataclasses.replace(SEQ_SMALL, input_dim=128, n_layers=1, max_steps=6, slots=8)
    w = weights(cfg)
    rng = np.random.default_rng(77)
    w["ln_in_g"] = rng.uniform(0.1, 3.0, cfg.input_dim).astype(np.float32)
    w["ln_in_b"] = rng.normal(0.0, 1.0, cfg.input_dim).astype(np.float32)
    gpu = Scorer(w, n_heads=cfg.n_heads, max_steps=cfg.max_steps, max_traces=cfg.slots)
    hist = {t: [] for t in range(cfg.slots)}
    for r in range(cfg.max_steps):
        ids = list(range(cfg.slots)) if r % 2 == 0 else [1, 6, 3]
        x = 4.0 + 0.5 * bf16_to_f64(step_states(cfg, r)[ids])
        H = to_bf16_bits(x.astype(np.float32))
        got = gpu.step(ids, _bf16(H)).cpu().numpy()
        for i, t in enumerate(ids):
            hist[t].append(bf16_to_f64(H[i]))
            want = scorer_outputs(w, np.stack(hist[t]), cfg.n_heads)[-1]
            assert abs(got[i] - want) <= TOL, (r, t, got[i], want)
    gpu.check()


def test_wide_model_six_heads_three_output_splits():
    """d_model 384 (six heads): the reduces' column loops take a second pass
    past 256 columns, and W_o / W_2 split their K three ways (d_ff 384);
    every step against the oracle, a fork on the way."""
    import dataclasses
    cfg = dataclasses.replace(SEQ_SMALL, d_model=384, n_heads=6, d_ff=384, max_steps=10, slots=6)
    _, gpu, ref = _make(cfg)
    ids = [0, 1, 2, 3]
    for r in range(8):
        if r == 4:
            gpu.fork([2], [5])
            ref.fork([2], [5])
            ids = [0, 1, 2, 3, 5]
        H = step_states(cfg, r)[ids]
        got = gpu.step(ids, _bf16(H)).cpu().numpy()
        want = ref.step(ids, bf16_to_f64(H))
        assert float(np.abs(got - want).max()) <= TOL, r
    assert [gpu.steps(t) for t in range(cfg.slots)] == [len(h) for h in ref.hist]
    gpu.check()


def test_no_layers_and_single_step_capacity():
    """The scorer without Transformer layers (input LN, projection, GELU,
    output head) and a history capacity of one step."""
    import dataclasses
    cfg = dataclasses.replace(SEQ_SMALL, n_layers=0, max_steps=1, slots=5)
    w = weights(cfg)
    gpu = Scorer(w, n_heads=cfg.n_heads, max_steps=1, max_traces=cfg.slots)
    H = step_states(cfg, 3)[:5]
    got = gpu.step(list(range(5)), _bf16(H)).cpu().numpy()
    for t in range(5):
        assert abs(got[t] - scorer_outputs(w, bf16_to_f64(H[t:t + 1]), cfg.n_heads)[-1]) <= TOL
    with pytest.raises(GambitError):  # full
        gpu.step([0], _bf16(H[:1]))
    gpu.free([0])
    assert gpu.steps(0) == 0 and gpu.steps(1) == 1
    gpu.check()


def test_capacity_not_a_multiple_of_four_filled_with_forks():
    """A history capacity of 13 steps (the cache rounds each head's rows up to
    16): traces filled to capacity, a fork taken mid-way, every step against
    the oracle - the last group of four cached keys is partly past the end
    on most steps."""
    import dataclasses
    cfg = dataclasses.replace(SEQ_SMALL, max_steps=13, slots=6)
    _, gpu, ref = _make(cfg)
    ids = [0, 1, 2, 3]
    for r in range(cfg.max_steps):
        if r == 6:
            gpu.fork([1, 2], [4, 5])
            ref.fork([1, 2], [4, 5])
            ids = [0, 1, 2, 3, 4, 5]
        ids = [t for t in ids if len(ref.hist[t]) < cfg.max_steps]
        H = step_states(cfg, r)[ids]
        got = gpu.step(ids, _bf16(H)).cpu().numpy()
        want = ref.step(ids, bf16_to_f64(H))
        assert float(np.abs(got - want).max()) <= TOL, r
    assert [gpu.steps(t) for t in range(cfg.slots)] == [len(h) for h in ref.hist]
    assert gpu.steps(0) == cfg.max_steps
    gpu.check()


def test_histories_past_one_pass_of_the_attention_step():
    """Histories of up to 289 steps: the attention step scores 128 cached
    steps per pass and reads the values 128 steps at a time, so lengths
    just below, at and past 128 and 256 (and not multiples of four) take a
    second and a third pass; a fork at step 140 copies a long history."""
    import dataclasses
    cfg = dataclasses.replace(SEQ_SMALL, max_steps=300, slots=4)
    w, gpu, _ = _make(cfg)
    hist = {t: [] for t in range(cfg.slots)}
    ids = [0, 1, 2]
    check = {0, 126, 127, 128, 129, 131, 141, 200, 255, 256, 257, 260, 288}
    for r in range(289):
        if r == 140:
            gpu.fork([1], [3])
            hist[3] = list(hist[1])
            ids = [0, 1, 2, 3]
        H = step_states(cfg, r)[ids]
        got = gpu.step(ids, _bf16(H)).cpu().numpy()
        for i, t in enumerate(ids):
            hist[t].append(bf16_to_f64(H[i]))
        if r in check:
            for i, t in enumerate(ids):
                want = scorer_outputs(w, np.stack(hist[t]), cfg.n_heads)[-1]
                assert abs(got[i] - want) <= TOL, (r, t, got[i], want)
    assert [gpu.steps(t) for t in range(cfg.slots)] == [289, 289, 289, 289]  # the fork copied 140 steps
    gpu.check()
