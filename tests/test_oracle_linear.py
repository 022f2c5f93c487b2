"""Pins for the oracle's linear-attention variant (no GPU).

The deployment the paper describes serves the evaluator with linear attention (Appendix B.3),
the kernelized form of the cited linear-attention work: weights phi(q) . phi(k) with
phi = elu + 1, normalised by their sum.  These tests check the oracle's spelling of it against
a hand-worked instance, closed forms, the scalar brute-force form, the associativity identity
that turns the context keys/values into a fixed-size state (the variant's key/value cache),
exact reuse (cached == naive) and the set-wise invariants of Section 4.4.
"""
import json
import math
import os

import numpy as np
import pytest

import gen
import oracle
from oracle import evaluator as ev


def _rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


def _golden():
    with open(os.path.join(os.path.dirname(__file__), "golden", "linear_attention_example.json")) as f:
        return json.load(f)


@pytest.fixture(scope="module")
def cfg0_lin():
    c = gen.config(0, attention="linear")
    return c, gen.make_weights(c), gen.make_inputs(c)


@pytest.fixture(scope="module")
def cfg1_lin_small():
    c = gen.config(1, K=6, B=2, T=40, attention="linear")
    return c, gen.make_weights(c), gen.make_inputs(c)


# ------------------------------------------------------------------------ feature map, closed forms

def test_feature_map_values():
    phi = oracle.elu_plus_one
    assert phi(np.array(0.0)) == 1.0
    assert phi(np.array(1.0)) == 2.0
    assert phi(np.array(2.5)) == 3.5
    assert phi(np.array(-1.0)) == math.exp(-1.0)
    assert phi(np.array(-30.0)) == math.exp(-30.0)
    # continuous at 0 from both sides, positive everywhere
    assert abs(phi(np.array(1e-12)) - phi(np.array(-1e-12))) < 3e-12
    assert np.all(phi(np.linspace(-50, 50, 1001)) > 0)


def test_hand_worked_instance():
    g = _golden()
    q = np.array([g["q"]])
    k, v = np.array(g["k"]), np.array(g["v"])
    e1, e2 = math.exp(-1.0), math.exp(-2.0)
    w1, w2 = 3.0 + e1, 1.5 * e2 + 4.0 * e1          # the derivation's closed forms
    assert abs(w1 - g["weights"][0]) < 1e-15 and abs(w2 - g["weights"][1]) < 1e-15
    want = np.array([[2 * w1, 4 * w2 - w1]]) / (w1 + w2)
    assert _rel(want, [g["out"]]) < 1e-15
    assert _rel(oracle.linear_attention(q, k, v, 1), want) < 1e-15
    st = oracle.linear_kv_state(k, v, 1)[0]
    fq = oracle.elu_plus_one(q[0])
    assert _rel((fq @ st[:2]) / (fq @ st[2]), want[0]) < 1e-15


@pytest.mark.parametrize("mistake", ["relu_plus_one", "no_normaliser", "scaled", "softmax", "phi_on_values"])
def test_planted_mistakes_miss_the_hand_worked_instance(mistake):
    """Plausible misreadings of the variant, planted in a copy of the oracle's formula, each
    disagree with the hand-worked instance."""
    g = _golden()
    q, k, v = np.array([g["q"]]), np.array(g["k"]), np.array(g["v"])
    phi = oracle.elu_plus_one
    if mistake == "relu_plus_one":
        w = (np.maximum(q, 0) + 1) @ (np.maximum(k, 0) + 1).T
        out = (w @ v) / w.sum(1, keepdims=True)
    elif mistake == "no_normaliser":
        out = (phi(q) @ phi(k).T) @ v
    elif mistake == "scaled":
        w = phi(q / math.sqrt(2)) @ phi(k / math.sqrt(2)).T
        out = (w @ v) / w.sum(1, keepdims=True)
    elif mistake == "softmax":
        out = oracle.attention(q, k, v, 1)
    else:
        w = phi(q) @ phi(k).T
        out = (w @ phi(v)) / w.sum(1, keepdims=True)
    assert _rel(out, [g["out"]]) > 1e-3


def test_single_key_returns_value():
    rng = np.random.default_rng(21)
    q = rng.standard_normal((5, 8))
    k, v = rng.standard_normal((1, 8)), rng.standard_normal((1, 8))
    assert np.allclose(oracle.linear_attention(q, k, v, 2), np.broadcast_to(v, (5, 8)), rtol=0, atol=1e-15)


def test_identical_keys_give_mean_of_values():
    rng = np.random.default_rng(22)
    q = rng.standard_normal((4, 12))
    k = np.broadcast_to(rng.standard_normal((1, 12)), (9, 12))
    v = rng.standard_normal((9, 12))
    out = oracle.linear_attention(q, k, v, 3)
    assert np.allclose(out, np.broadcast_to(v.mean(0), out.shape), rtol=0, atol=1e-14)


def test_zero_query_weights_keys_by_feature_sum():
    """q = 0 gives phi(q) = 1, so key j weighs sum_i phi(k_j)_i, the same for every query."""
    rng = np.random.default_rng(23)
    k, v = rng.standard_normal((7, 4)), rng.standard_normal((7, 4))
    w = np.exp(np.minimum(k, 0)) * (k <= 0) + (k + 1) * (k > 0)
    s = w.sum(1)
    want = (s @ v) / s.sum()
    out = oracle.linear_attention(np.zeros((3, 4)), k, v, 1)
    assert np.allclose(out, np.broadcast_to(want, out.shape), rtol=0, atol=1e-14)


def test_key_order_does_not_matter():
    rng = np.random.default_rng(24)
    q, k, v = rng.standard_normal((6, 16)), rng.standard_normal((11, 16)), rng.standard_normal((11, 16))
    p = rng.permutation(11)
    assert _rel(oracle.linear_attention(q, k[p], v[p], 2), oracle.linear_attention(q, k, v, 2)) < 1e-13


def test_state_form_equals_definition():
    """The fixed-size state (sum of phi(k) v^T and of phi(k) per head) reproduces the defining
    form for any query: the reassociation behind the variant's key/value cache."""
    rng = np.random.default_rng(25)
    H, dh, T = 4, 8, 37
    q, k, v = (rng.standard_normal((n, H * dh)) for n in (13, T, T))
    st = oracle.linear_kv_state(k, v, H)
    assert st.shape == (H, dh + 1, dh)
    want = oracle.linear_attention(q, k, v, H)
    for h in range(H):
        fq = oracle.elu_plus_one(q[:, h * dh:(h + 1) * dh])
        got = (fq @ st[h, :dh]) / (fq @ st[h, dh])[:, None]
        assert _rel(got, want[:, h * dh:(h + 1) * dh]) < 1e-12


def test_module_kinds():
    c = gen.config(0, attention="linear")
    assert [ev.module_attention(c, m) for m in ("ctx", "item_self", "item_cross", "seq", "cross")] == \
        ["linear", "softmax", "linear", "softmax", "linear"]
    assert {ev.module_attention(gen.config(0), m) for m in ("ctx", "item_self", "item_cross", "seq", "cross")} == \
        {"softmax"}


# ------------------------------------------------------------------------ whole pass

def test_brute_force_linear_cfg0(cfg0_lin):
    c, W, I = cfg0_lin
    o = oracle.evaluate_naive(c, W, I)[0]
    br = oracle.evaluate_brute(c, W, I, 0)
    assert _rel(o["c"], br["c"]) < 1e-12
    assert _rel(o["Cp"], br["Cp"]) < 1e-12
    assert _rel(o["scores"], br["scores"]) < 1e-12
    assert o["best"] == br["best"]


def test_brute_force_linear_two_heads_two_layers():
    c = gen.config(0, n_heads=2, n_layers=2, K=3, L=4, attention="linear")
    W, I = gen.make_weights(c), gen.make_inputs(c)
    o = oracle.evaluate_cached(c, W, I)[0]
    br = oracle.evaluate_brute(c, W, I, 0)
    assert _rel(o["scores"], br["scores"]) < 1e-12


def test_linear_variant_changes_the_attention(cfg0_lin):
    """The variant swaps the attention itself: a context block's attention output differs by
    percents (with N(0, 0.02) projections every weight is near uniform); through the small output
    projections and the residual stream the scores move much less."""
    c, W, I = cfg0_lin
    d = c.d
    x = ev.layer_norm(np.asarray(I["x"][0], np.float64), W["ctx.0.ln1.g"], W["ctx.0.ln1.b"])
    qkv = x @ np.asarray(W["ctx.0.wqkv"], np.float64) + W["ctx.0.bqkv"]
    q, k, v = qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:]
    assert _rel(ev.attend(q, k, v, c.n_heads, "linear"), ev.attend(q, k, v, c.n_heads, "softmax")) > 1e-2
    lin = oracle.evaluate_cached(c, W, I)[0]["scores"]
    soft = oracle.evaluate_cached(gen.config(0), W, I)[0]["scores"]
    assert _rel(lin, soft) > 1e-7


def test_cached_equals_naive_linear(cfg0_lin, cfg1_lin_small):
    for c, W, I in (cfg0_lin, cfg1_lin_small):
        reqs = list(range(c.B))
        n = oracle.evaluate_naive(c, W, I, requests=reqs)
        ca = oracle.evaluate_cached(c, W, I, requests=reqs)
        for b in reqs:
            assert _rel(n[b]["scores"], ca[b]["scores"]) < 1e-12
            assert n[b]["best"] == ca[b]["best"]


def test_linear_scores_permutation_equivariant(cfg1_lin_small):
    c, W, I = cfg1_lin_small
    perm = np.random.default_rng(26).permutation(c.K)
    J = dict(I)
    J["lists"] = I["lists"][:, perm]
    a = oracle.evaluate_cached(c, W, I, requests=[1])[1]
    b = oracle.evaluate_cached(c, W, J, requests=[1])[1]
    assert _rel(b["scores"], a["scores"][perm]) < 1e-12
    assert perm[b["best"]] == a["best"]
