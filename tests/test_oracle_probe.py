"""Pins of the oracle's probe, ranking and prune/branch plan."""
import math

import numpy as np
import pytest
import torch

from oracle.probe import probe_scores, prune_branch_plan, rank, sigmoid


def test_zero_weights_give_one_half():
    h = np.random.default_rng(0).standard_normal((5, 64))
    assert (probe_scores(h, np.zeros(64), 0.0) == 0.5).all()


def test_unit_vector_picks_one_weight():
    rng = np.random.default_rng(1)
    w, b = rng.standard_normal(16), 0.25
    for i in range(16):
        e = np.zeros((1, 16))
        e[0, i] = 1.0
        assert probe_scores(e, w, b)[0] == pytest.approx(1 / (1 + math.exp(-(w[i] + b))), abs=1e-15)


def test_sigmoid_closed_forms():
    assert sigmoid(np.array([0.0]))[0] == 0.5
    assert sigmoid(np.array([math.log(3.0)]))[0] == pytest.approx(0.75, abs=1e-15)
    z = np.linspace(-30, 30, 301)
    assert np.abs(sigmoid(z) + sigmoid(-z) - 1).max() < 1e-15


def test_matches_torch_sigmoid_of_matvec():
    rng = np.random.default_rng(2)
    h, w = rng.standard_normal((40, 4096)), rng.standard_normal(4096) / 64
    ref = torch.sigmoid(torch.from_numpy(h) @ torch.from_numpy(w) + 0.1).numpy()
    assert np.abs(probe_scores(h, w, 0.1) - ref).max() < 1e-14


def test_rank_breaks_ties_by_lowest_id():
    assert rank([3, 1, 0, 2], [0.5, 0.7, 0.5, 0.7]) == [1, 2, 0, 3]
    assert rank([9, 4, 6], [0.1, 0.1, 0.1]) == [4, 6, 9]
    assert rank([5, 2, 8], [0.2, 0.9, 0.4]) == [2, 8, 5]


def test_case2_swap_is_one_to_one():
    """Eq. 3: prune the bottom K, branch the top K, one child each."""
    ids = list(range(8))
    scores = [0.1, 0.9, 0.3, 0.8, 0.2, 0.7, 0.6, 0.05]
    order = rank(ids, scores)            # 1, 3, 5, 6, 2, 4, 0, 7
    K = 2
    freed, pairs = prune_branch_plan(ids, order[:8 - K], K)
    assert freed == [0, 7]
    assert pairs == [(0, 1), (7, 3)]


def test_fanout_plan_keeps_population_size():
    n, keep, npar = 64, 16, 16
    rng = np.random.default_rng(3)
    ids = list(rng.permutation(200)[:n])
    scores = rng.random(n)
    kp = rank(ids, scores)[:keep]
    freed, pairs = prune_branch_plan(ids, kp, npar)
    assert freed == sorted(set(ids) - set(kp))
    assert [c for c, _ in pairs] == freed
    # zero-sum: kept + children = population; each parent gets (n-keep)/npar children
    assert len(kp) + len(pairs) == n
    per = {}
    for j, (_, p) in enumerate(pairs):
        per[p] = per.get(p, 0) + 1
        assert p == kp[j // 3]
    assert sorted(per) == sorted(kp[:npar]) and set(per.values()) == {3}


def test_plan_rejects_bad_shapes():
    with pytest.raises(ValueError):
        prune_branch_plan([0, 1, 2, 3], [0, 1], 3)
    with pytest.raises(ValueError):
        prune_branch_plan([0, 1, 2, 3], [0, 1, 2], 0)
