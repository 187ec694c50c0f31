"""Pins of the oracle's 2-layer MLP scorer: closed forms (zero first layer,
one hidden unit, activation values) and torch's own Linear -> act -> Linear
-> sigmoid in float64 on the same weights (an independent library)."""
import math

import numpy as np
import pytest
import torch

from oracle.mlp import activation, mlp_logits, mlp_scores


@pytest.mark.parametrize("act", ["relu", "gelu"])
def test_matches_torch_sequential(act):
    rng = np.random.default_rng(5)
    n, Dh, H1 = 7, 64, 32
    h = rng.standard_normal((n, Dh))
    W1 = rng.standard_normal((H1, Dh)) / 8
    b1 = rng.standard_normal(H1) / 4
    w2 = rng.standard_normal(H1) / 5
    b2 = 0.3
    lin1 = torch.nn.Linear(Dh, H1).double()
    lin2 = torch.nn.Linear(H1, 1).double()
    with torch.no_grad():
        lin1.weight.copy_(torch.from_numpy(W1))
        lin1.bias.copy_(torch.from_numpy(b1))
        lin2.weight.copy_(torch.from_numpy(w2[None]))
        lin2.bias.fill_(b2)
    a = torch.nn.ReLU() if act == "relu" else torch.nn.GELU(approximate="none")
    with torch.no_grad():
        want = torch.sigmoid(lin2(a(lin1(torch.from_numpy(h))))).squeeze(1).numpy()
    got = mlp_scores(h, W1, b1, w2, b2, act)
    assert np.abs(got - want).max() < 1e-14


def test_zero_first_layer_is_a_constant():
    rng = np.random.default_rng(1)
    h = rng.standard_normal((4, 16))
    b1 = np.array([1.0, -2.0, 0.5])
    w2 = np.array([0.25, 3.0, -1.0])
    z = mlp_logits(h, np.zeros((3, 16)), b1, w2, 0.1, "relu")
    assert np.allclose(z, 0.25 * 1.0 + 0.0 * 3.0 - 1.0 * 0.5 + 0.1, atol=0, rtol=0)


def test_one_hidden_unit():
    h = np.array([[1.0, 2.0], [-3.0, 1.0]])
    z = mlp_logits(h, np.array([[0.5, 1.0]]), np.array([0.0]), np.array([2.0]), -1.0, "relu")
    assert z.tolist() == [2.0 * 2.5 - 1.0, -1.0]       # relu(0.5 + 2) and relu(-0.5)
    assert mlp_scores(h, np.array([[0.0, 0.0]]), np.array([0.0]), np.array([1.0]), 0.0, "relu").tolist() == [0.5, 0.5]


def test_activation_values():
    x = np.array([-2.0, 0.0, 1.0])
    assert activation(x, "relu").tolist() == [0.0, 0.0, 1.0]
    g = activation(x, "gelu")
    assert g[1] == 0.0
    assert abs(g[2] - 0.5 * (1 + math.erf(1 / math.sqrt(2)))) < 1e-15    # x * Phi(x) at 1
    assert abs(g[0] + 2 * 0.5 * (1 - math.erf(2 / math.sqrt(2)))) < 1e-15  # gelu(-x) = -x * Phi(-x)
