"""Pins of the sequence-scorer oracle (App. A.1, Eqs. 4-6).

* LayerNorm, GELU and SiLU against torch's library functions in float64.
* RoPE: position 0 is the identity; every rotated pair keeps its norm; the
  angle of pair i at position p is p * 10000^(-2i/hd) (unit vectors, closed
  form); scores depend only on the position difference.
* Causal multi-head attention against torch's scaled_dot_product_attention
  (is_causal) on the same rotated queries and keys.
* SwiGLU on a 1 x 1 model by hand; a zero gate gives zero.
* The whole scorer: with no layers it is LN -> W_in -> GELU -> LN -> w_out
  -> sigmoid by torch's functions; y_t does not depend on later steps; at one
  step the queries and keys do not matter (attention over one position
  returns its value); the history model's fork equals a copy.
* The layer stacking (residuals, pre-norm order, attention before the
  feed-forward, layers in order) against torch's nn.TransformerEncoderLayer
  with norm_first=True: with zero queries over several steps (uniform causal
  weights, so the rotary embedding plays no part) and with the full weights
  at one step.
"""
import math

import numpy as np
import torch
import torch.nn.functional as F

from oracle.seqscorer import (LN_EPS, SeqScorerModel, causal_mha, gelu, layer_norm, rope, scorer_outputs,
                              silu, swiglu)

RNG = np.random.default_rng(5)


def _w(cfg_layers=1, D=24, d=16, f=20):
    r = np.random.default_rng(7)
    lin = lambda o, i: r.standard_normal((o, i)) / math.sqrt(i)  # noqa: E731
    w = {"ln_in_g": 1 + 0.1 * r.standard_normal(D), "ln_in_b": 0.1 * r.standard_normal(D), "W_in": lin(d, D),
         "ln_out_g": 1 + 0.1 * r.standard_normal(d), "ln_out_b": 0.1 * r.standard_normal(d),
         "w_out": r.standard_normal(d) / math.sqrt(d), "layers": []}
    for _ in range(cfg_layers):
        w["layers"].append({"ln1_g": 1 + 0.1 * r.standard_normal(d), "ln1_b": 0.1 * r.standard_normal(d),
                            "Wq": lin(d, d), "Wk": lin(d, d), "Wv": lin(d, d), "Wo": lin(d, d),
                            "ln2_g": 1 + 0.1 * r.standard_normal(d), "ln2_b": 0.1 * r.standard_normal(d),
                            "W1": lin(f, d), "W3": lin(f, d), "W2": lin(d, f)})
    return w


def test_layer_norm_gelu_silu_match_torch():
    x = RNG.standard_normal((5, 33)) * 3 + 1
    g, b = RNG.standard_normal(33), RNG.standard_normal(33)
    ref = F.layer_norm(torch.from_numpy(x), (33,), torch.from_numpy(g), torch.from_numpy(b), eps=LN_EPS).numpy()
    assert np.allclose(layer_norm(x, g, b), ref, rtol=0, atol=1e-12)
    assert np.allclose(gelu(x), F.gelu(torch.from_numpy(x)).numpy(), rtol=0, atol=1e-13)
    assert np.allclose(silu(x), F.silu(torch.from_numpy(x)).numpy(), rtol=0, atol=1e-13)


def test_rope_closed_forms_and_relative_positions():
    hd = 8
    x = RNG.standard_normal((6, hd))
    assert np.array_equal(rope(x, np.zeros(6)), x)
    y = rope(x, np.arange(6) * 3.7)
    for i in range(hd // 2):  # each pair keeps its norm
        assert np.allclose(np.hypot(y[:, i], y[:, i + hd // 2]), np.hypot(x[:, i], x[:, i + hd // 2]))
    # unit vector e_i at position p: (cos, sin) of p * 10000^(-2i/hd) in components i, i + hd/2
    for i in range(hd // 2):
        e = np.zeros((1, hd))
        e[0, i] = 1
        ang = 5.0 * 10000.0 ** (-2 * i / hd)
        r = rope(e, np.array([5.0]))[0]
        assert abs(r[i] - math.cos(ang)) < 1e-15 and abs(r[i + hd // 2] - math.sin(ang)) < 1e-15
    # q_m . k_n depends on m - n only
    q, k = RNG.standard_normal((1, hd)), RNG.standard_normal((1, hd))
    for m, n, s in [(3, 1, 7), (0, 5, 11), (9, 9, 2)]:
        a = rope(q, np.array([m])) @ rope(k, np.array([n])).T
        b = rope(q, np.array([m + s])) @ rope(k, np.array([n + s])).T
        assert abs(a - b).max() < 1e-12


def test_causal_mha_matches_torch_sdpa():
    T, d, H = 7, 16, 4
    hd = d // H
    x = RNG.standard_normal((T, d))
    Wq, Wk, Wv, Wo = (RNG.standard_normal((d, d)) / 4 for _ in range(4))
    q, k, v = x @ Wq.T, x @ Wk.T, x @ Wv.T
    pos = np.arange(T)
    qs = np.stack([rope(q[:, h * hd:(h + 1) * hd], pos) for h in range(H)])
    ks = np.stack([rope(k[:, h * hd:(h + 1) * hd], pos) for h in range(H)])
    vs = np.stack([v[:, h * hd:(h + 1) * hd] for h in range(H)])
    o = F.scaled_dot_product_attention(torch.from_numpy(qs), torch.from_numpy(ks), torch.from_numpy(vs),
                                       is_causal=True).numpy()
    ref = np.concatenate(list(o), axis=1) @ Wo.T
    assert np.allclose(causal_mha(x, Wq, Wk, Wv, Wo, H), ref, rtol=0, atol=1e-12)


def test_swiglu_by_hand():
    a, b, c, x = 0.7, -1.3, 2.1, 0.9
    want = c * (a * x / (1 + math.exp(-a * x))) * (b * x)
    got = swiglu(np.array([[x]]), np.array([[a]]), np.array([[b]]), np.array([[c]]))[0, 0]
    assert abs(got - want) < 1e-15
    z = swiglu(RNG.standard_normal((3, 4)), np.zeros((5, 4)), RNG.standard_normal((5, 4)),
               RNG.standard_normal((4, 5)))
    assert (z == 0).all()


def test_scorer_without_layers_matches_torch():
    w = _w(cfg_layers=0)
    H = RNG.standard_normal((4, 24))
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))  # noqa: E731
    x = F.gelu(F.linear(F.layer_norm(t(H), (24,), t(w["ln_in_g"]), t(w["ln_in_b"]), eps=LN_EPS), t(w["W_in"])))
    y = torch.sigmoid(F.layer_norm(x, (16,), t(w["ln_out_g"]), t(w["ln_out_b"]), eps=LN_EPS) @ t(w["w_out"]))
    assert np.allclose(scorer_outputs(w, H, 4), y.numpy(), rtol=0, atol=1e-14)


def test_causality_and_single_step():
    w = _w(cfg_layers=2)
    H = RNG.standard_normal((9, 24))
    y = scorer_outputs(w, H, 4)
    for t in range(1, 9):
        assert np.allclose(scorer_outputs(w, H[:t], 4), y[:t], rtol=0, atol=1e-14)
        H2 = H.copy()
        H2[t:] = RNG.standard_normal((9 - t, 24))
        assert np.allclose(scorer_outputs(w, H2, 4)[:t], y[:t], rtol=0, atol=1e-14)
        assert abs(scorer_outputs(w, H2, 4)[t] - y[t]) > 1e-9  # the new step does matter
    w2 = _w(cfg_layers=2)
    for L in w2["layers"]:
        L["Wq"], L["Wk"] = RNG.standard_normal((16, 16)), RNG.standard_normal((16, 16))
    assert abs(scorer_outputs(w2, H[:1], 4)[0] - y[0]) < 1e-14


def test_history_model_fork_is_a_copy():
    w = _w(cfg_layers=1)
    m = SeqScorerModel(w, 4, slots=4, max_steps=10)
    H = RNG.standard_normal((6, 24))
    for s in range(3):
        m.step([0, 1], H[s:s + 2])
    m.fork([0], [2])
    a = m.step([0], H[5:6])[0]
    b = m.step([2], H[5:6])[0]
    assert a == b
    m.free([1])
    assert m.step([1], H[:1])[0] == scorer_outputs(w, H[:1], 4)[0]


def _torch_stack(w, H, n_heads, causal=True):
    """The scorer's layers run by torch's own pre-norm encoder layers
    (nn.TransformerEncoderLayer with norm_first=True: x + SA(LN1(x)), then
    x + FF(LN2(x))).  The gated feed-forward is expressed in torch's
    Linear -> activation -> Linear form: linear1 stacks W1 over W3, the
    activation multiplies SiLU of the first half by the second half (padded
    back with zeros) and linear2 is [W2 | 0]."""
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))  # noqa: E731
    d = w["W_in"].shape[0]
    f = w["layers"][0]["W1"].shape[0] if w["layers"] else 1

    def gated(z):
        return torch.cat([F.silu(z[..., :f]) * z[..., f:], torch.zeros_like(z[..., f:])], dim=-1)

    x = F.gelu(F.linear(F.layer_norm(t(H), (H.shape[1],), t(w["ln_in_g"]), t(w["ln_in_b"]), eps=LN_EPS),
                        t(w["W_in"])))[None]
    for L in w["layers"]:
        lay = torch.nn.TransformerEncoderLayer(d, n_heads, dim_feedforward=2 * f, dropout=0.0, activation=gated,
                                               layer_norm_eps=LN_EPS, batch_first=True, norm_first=True, dtype=torch.float64)
        with torch.no_grad():
            for b in (lay.self_attn.in_proj_bias, lay.self_attn.out_proj.bias, lay.linear1.bias, lay.linear2.bias):
                b.zero_()  # the scorer's linear maps have no biases
            lay.self_attn.in_proj_weight.copy_(t(np.concatenate([L["Wq"], L["Wk"], L["Wv"]])))
            lay.self_attn.out_proj.weight.copy_(t(L["Wo"]))
            lay.linear1.weight.copy_(t(np.concatenate([L["W1"], L["W3"]])))
            lay.linear2.weight.copy_(t(np.concatenate([L["W2"], np.zeros_like(L["W2"])], axis=1)))
            lay.norm1.weight.copy_(t(L["ln1_g"]))
            lay.norm1.bias.copy_(t(L["ln1_b"]))
            lay.norm2.weight.copy_(t(L["ln2_g"]))
            lay.norm2.bias.copy_(t(L["ln2_b"]))
        lay.train()  # the reference (non-fused) code path; dropout is 0
        T = x.shape[1]
        mask = torch.nn.Transformer.generate_square_subsequent_mask(T, dtype=torch.float64) if causal else None
        with torch.no_grad():
            x = lay(x, src_mask=mask, is_causal=causal)
    y = torch.sigmoid(F.layer_norm(x[0], (d,), t(w["ln_out_g"]), t(w["ln_out_b"]), eps=LN_EPS) @ t(w["w_out"]))
    return y.numpy()


def test_layer_stacking_matches_torch_pre_norm_encoder():
    """Residuals and the pre-norm order of each layer (App. A.1's Transformer
    over the step sequence), pinned by torch's own encoder layer.  Queries are
    zero, so every causal position averages the values of steps 0..t equally
    and the rotary embedding (pinned separately) plays no part: what is left
    is the layer structure - LN1 before attention, LN2 before the gated
    feed-forward, both added back to the stream, attention before the
    feed-forward, layers in order.  A dropped residual or a post-norm layer
    (LN after the addition) fails it."""
    for n_layers, T in [(1, 1), (1, 2), (2, 5), (3, 7)]:
        w = _w(cfg_layers=n_layers)
        for L in w["layers"]:
            L["Wq"] = np.zeros_like(L["Wq"])
        H = RNG.standard_normal((T, 24))
        ref = _torch_stack(w, H, 4)
        got = scorer_outputs(w, H, 4)
        assert np.allclose(got, ref, rtol=0, atol=1e-13), (n_layers, T, got, ref)


def test_layer_stacking_one_step_full_weights():
    """At a single step attention returns the step's own value (any queries
    and keys; the rotation at position 0 is the identity), so torch's
    pre-norm encoder layer with the full weights gives the scorer's output."""
    w = _w(cfg_layers=2)
    H = RNG.standard_normal((1, 24))
    assert np.allclose(scorer_outputs(w, H, 4), _torch_stack(w, H, 4, causal=False), rtol=0, atol=1e-13)
