"""Pins of the oracle's decode attention.

Each check is fixed by mathematics or by an independent library routine:
closed forms (L = 1, equal keys, zero scale, a dominant key), the softmax
invariant sum p = 1, permutation invariance over context positions, the
log-sum-exp split identity, and agreement with PyTorch's causal
scaled_dot_product_attention in float64 when one trace is decoded token by
token (which pins the scale, the grouped-head mapping h -> h // g and the
inclusion of the current token).
"""
import math

import numpy as np
import pytest
import torch

from oracle.attention import decode_attention, softmax_weights

D = 128


def _rand(rng, *shape):
    return rng.standard_normal(shape)


def test_single_token_returns_its_value():
    rng = np.random.default_rng(0)
    q, K, V = _rand(rng, 8, D), _rand(rng, 1, 2, D), _rand(rng, 1, 2, D)
    o = decode_attention(q, K, V, 1 / math.sqrt(D))
    for h in range(8):
        assert np.array_equal(o[h], V[0, h // 4])


@pytest.mark.parametrize("kind", ["equal_keys", "zero_query", "zero_scale"])
def test_uniform_weights_give_mean_of_values(kind):
    rng = np.random.default_rng(1)
    L, Hq, Hkv = 37, 8, 2
    q, K, V = _rand(rng, Hq, D), _rand(rng, L, Hkv, D), _rand(rng, L, Hkv, D)
    scale = 1 / math.sqrt(D)
    if kind == "equal_keys":
        K[:] = K[0]
    elif kind == "zero_query":
        q[:] = 0
    else:
        scale = 0.0
    o = decode_attention(q, K, V, scale)
    for h in range(Hq):
        assert np.allclose(o[h], V[:, h // 4].mean(axis=0), rtol=0, atol=1e-13)


def test_dominant_key_selects_its_value():
    rng = np.random.default_rng(2)
    L, Hq, Hkv = 20, 4, 1
    q, K, V = _rand(rng, Hq, D), _rand(rng, L, Hkv, D) * 0.01, _rand(rng, L, Hkv, D)
    K[7, 0] = 50.0 * q[0] / np.linalg.norm(q[0])
    o = decode_attention(q[:1], K, V, 1.0)
    assert np.allclose(o[0], V[7, 0], atol=1e-12)


def test_weights_sum_to_one_and_are_positive():
    rng = np.random.default_rng(3)
    q, K = _rand(rng, 32, D) * 3, _rand(rng, 999, 8, D) * 3
    p = softmax_weights(q, K, 1 / math.sqrt(D))
    assert (p > 0).all()
    assert np.abs(p.sum(axis=1) - 1).max() < 1e-12


def test_permutation_invariance():
    rng = np.random.default_rng(4)
    L = 300
    q, K, V = _rand(rng, 32, D), _rand(rng, L, 8, D), _rand(rng, L, 8, D)
    perm = rng.permutation(L)
    a = decode_attention(q, K, V, 0.1)
    b = decode_attention(q, K[perm], V[perm], 0.1)
    assert np.abs(a - b).max() < 1e-13


def test_log_sum_exp_split_identity():
    """Attention over [A; B] = Z-weighted mix of attention over A and over B."""
    rng = np.random.default_rng(5)
    q, K, V = _rand(rng, 8, D), _rand(rng, 200, 2, D), _rand(rng, 200, 2, D)
    s = 1 / math.sqrt(D)
    cut = 77
    full = decode_attention(q, K, V, s)
    oa = decode_attention(q, K[:cut], V[:cut], s)
    ob = decode_attention(q, K[cut:], V[cut:], s)
    for h in range(8):
        za = np.exp(K[:cut, h // 4] @ q[h] * s).sum()
        zb = np.exp(K[cut:, h // 4] @ q[h] * s).sum()
        mix = (za * oa[h] + zb * ob[h]) / (za + zb)
        assert np.abs(mix - full[h]).max() < 1e-12


@pytest.mark.parametrize("Hq,Hkv", [(32, 8), (64, 8), (8, 2), (4, 4)])
def test_token_by_token_matches_torch_causal_sdpa(Hq, Hkv):
    rng = np.random.default_rng(6)
    L = 45
    Q, K, V = _rand(rng, L, Hq, D), _rand(rng, L, Hkv, D), _rand(rng, L, Hkv, D)
    scale = 1 / math.sqrt(D)
    g = Hq // Hkv
    tq = torch.from_numpy(Q).permute(1, 0, 2)[None]                       # [1][Hq][L][D]
    tk = torch.from_numpy(K).permute(1, 0, 2).repeat_interleave(g, 0)[None]
    tv = torch.from_numpy(V).permute(1, 0, 2).repeat_interleave(g, 0)[None]
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True,
                                                           scale=scale)[0].permute(1, 0, 2).numpy()
    for i in range(L):
        o = decode_attention(Q[i], K[:i + 1], V[:i + 1], scale)
        assert np.abs(o - ref[i]).max() < 1e-12, i


def test_head_mapping_is_consecutive_groups():
    """Query heads 0..g-1 read KV head 0, g..2g-1 read KV head 1 (not h % Hkv)."""
    rng = np.random.default_rng(7)
    L, Hq, Hkv = 10, 8, 2
    q, K = _rand(rng, Hq, D), _rand(rng, L, Hkv, D)
    V = np.zeros((L, Hkv, D))
    V[:, 0], V[:, 1] = 1.0, -1.0
    o = decode_attention(q, K, V, 0.1)
    assert np.abs(o[:4] - 1.0).max() < 1e-14 and np.abs(o[4:] + 1.0).max() < 1e-14


def test_empty_context_rejected():
    with pytest.raises(ValueError):
        decode_attention(np.zeros((4, D)), np.zeros((0, 1, D)), np.zeros((0, 1, D)), 1.0)


def _brute_force(q, K, V, scale):
    """Scalar loops over Python floats and math.exp, straight from the
    definition (no max subtraction, no library linear algebra)."""
    Hq, L, Hkv, Dd = len(q), len(K), len(K[0]), len(q[0])
    g = Hq // Hkv
    out = []
    for h in range(Hq):
        w = []
        for j in range(L):
            dot = 0.0
            for d in range(Dd):
                dot += q[h][d] * K[j][h // g][d]
            w.append(math.exp(scale * dot))
        z = sum(w)
        out.append([sum(w[j] * V[j][h // g][d] for j in range(L)) / z for d in range(Dd)])
    return out


@pytest.mark.parametrize("L,Hq,Hkv,Dd", [(1, 2, 1, 3), (2, 4, 2, 5), (5, 8, 2, 4), (7, 6, 3, 2), (9, 4, 4, 8)])
def test_matches_scalar_brute_force_on_tiny_inputs(L, Hq, Hkv, Dd):
    rng = np.random.default_rng(100 + L)
    q, K, V = _rand(rng, Hq, Dd), _rand(rng, L, Hkv, Dd), _rand(rng, L, Hkv, Dd)
    scale = 0.7
    ref = np.array(_brute_force(q.tolist(), K.tolist(), V.tolist(), scale))
    o = decode_attention(q, K, V, scale)
    assert np.abs(o - ref).max() < 1e-12
