"""Pins for the CPU oracle (no GPU).

Each test checks the oracle against something other than itself: torch's
library transformer layers, the scalar brute-force form, closed forms of
attention and LayerNorm, and the invariants the paper's construction fixes
(exact reuse in Section 4.2, positions after indexing in Section 4.3, a
set-wise cross-sequence module in Section 4.4, the argmax of eq. (1) with the
min-argmax tie rule of Appendix B.1).
"""
import numpy as np
import pytest
import torch

import gen
import oracle
from oracle import evaluator as ev
from tests.torch_reference import decoder_layer, encoder_layer, evaluate_torch


def _rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


@pytest.fixture(scope="module")
def cfg0():
    c = gen.config(0)
    return c, gen.make_weights(c), gen.make_inputs(c)


@pytest.fixture(scope="module")
def cfg1_small():
    """Workload-1 model with K=6 lists and two requests (the naive order stays cheap)."""
    c = gen.config(1, K=6, B=2)
    return c, gen.make_weights(c), gen.make_inputs(c)


# ----------------------------------------------------------------------------- library pins (P1)

@pytest.mark.parametrize("d,H,F,T", [(32, 1, 128, 7), (128, 4, 512, 33), (64, 2, 256, 9)])
def test_encoder_block_matches_torch_layer(d, H, F, T):
    c = gen.config(0, d=d, n_heads=H, ffn=F)
    W = gen.make_weights(c)
    x = np.random.default_rng(1).standard_normal((T, d))
    ours = ev.encoder_block(x, W, "seq.0", H)
    ref = encoder_layer(W, "seq.0", d, H, F)(torch.as_tensor(x)[None])[0].detach().numpy()
    assert _rel(ours, ref) < 1e-12


@pytest.mark.parametrize("d,H,F,U,T", [(32, 1, 128, 5, 16), (128, 4, 512, 21, 40)])
def test_item_layer_matches_torch_decoder_layer(d, H, F, U, T):
    c = gen.config(0, d=d, n_heads=H, ffn=F)
    W = gen.make_weights(c)
    rng = np.random.default_rng(2)
    G = rng.standard_normal((U, d))
    mem = rng.standard_normal((T, d))
    kv = [(mem @ W["ctx.kv.0.wk"].astype(np.float64) + W["ctx.kv.0.bk"],
           mem @ W["ctx.kv.0.wv"].astype(np.float64) + W["ctx.kv.0.bv"])]
    one_layer = gen.config(0, d=d, n_heads=H, ffn=F, n_layers=1)
    # the oracle's item encoder ends with item.lnf; apply the same LN to torch's layer output
    ours = ev.encode_items(one_layer, W, G, kv)
    out = decoder_layer(W, 0, d, H, F)(torch.as_tensor(G)[None], torch.as_tensor(mem)[None])[0]
    ref = ev.layer_norm(out.detach().numpy(), W["item.lnf.g"], W["item.lnf.b"])
    assert _rel(ours, ref) < 1e-12


def test_whole_pass_matches_torch_cfg0(cfg0):
    c, W, I = cfg0
    o = oracle.evaluate_cached(c, W, I, stages=True)[0]
    t = evaluate_torch(c, W, I, 0)
    for key in ("H", "c", "Cp", "scores"):
        assert _rel(o[key], t[key]) < 1e-12, key


def test_whole_pass_matches_torch_cfg1_slice(cfg1_small):
    c, W, I = cfg1_small
    o = oracle.evaluate_cached(c, W, I, requests=[1])[1]
    t = evaluate_torch(c, W, I, 1)
    assert _rel(o["Cp"], t["Cp"]) < 1e-12
    assert _rel(o["scores"], t["scores"]) < 1e-12


def test_whole_pass_matches_torch_text_shape():
    """Token-id context and items keyed on token id (workload-4 structure, tiny sizes)."""
    c = gen.config(4, B=1, T=12, d=64, n_heads=2, ffn=256, n_layers=2, K=3, L=6, M=50, vocab=50)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    o = oracle.evaluate_cached(c, W, I)[0]
    t = evaluate_torch(c, W, I, 0)
    assert _rel(o["scores"], t["scores"]) < 1e-12


# ----------------------------------------------------------------------------- brute force (P2)

def test_brute_force_cfg0(cfg0):
    c, W, I = cfg0
    o = oracle.evaluate_naive(c, W, I)[0]
    br = oracle.evaluate_brute(c, W, I, 0)
    assert _rel(o["c"], br["c"]) < 1e-12
    assert _rel(o["Cp"], br["Cp"]) < 1e-12
    assert _rel(o["scores"], br["scores"]) < 1e-12
    assert o["best"] == br["best"]


def test_brute_force_two_heads_two_layers():
    c = gen.config(0, n_heads=2, n_layers=2, K=3, L=4)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    o = oracle.evaluate_cached(c, W, I)[0]
    br = oracle.evaluate_brute(c, W, I, 0)
    assert _rel(o["scores"], br["scores"]) < 1e-12


# ----------------------------------------------------------------------------- exact reuse (P3)

def test_cached_equals_naive_cfg0(cfg0):
    c, W, I = cfg0
    n = oracle.evaluate_naive(c, W, I)[0]
    ca = oracle.evaluate_cached(c, W, I)[0]
    assert np.array_equal(n["scores"], ca["scores"]) or _rel(n["scores"], ca["scores"]) < 1e-12
    assert n["best"] == ca["best"]


def test_cached_equals_naive_cfg1_slice(cfg1_small):
    c, W, I = cfg1_small
    n = oracle.evaluate_naive(c, W, I, requests=[0, 1])
    ca = oracle.evaluate_cached(c, W, I, requests=[0, 1])
    for b in (0, 1):
        assert _rel(n[b]["scores"], ca[b]["scores"]) < 1e-12
        assert n[b]["best"] == ca[b]["best"]


# ----------------------------------------------------------------------------- integer steps (P4, P5, P6)

def test_distinct_items_matches_numpy_unique():
    rng = np.random.default_rng(3)
    for M, K, L in [(20, 4, 5), (200, 50, 10), (32000, 16, 64), (5, 7, 3)]:
        lists = rng.integers(0, M, (K, L))
        uniq, slot = oracle.distinct_items(lists)
        u_np, inv = np.unique(lists, return_inverse=True)
        assert np.array_equal(uniq, u_np)
        assert np.array_equal(slot.reshape(-1), inv.reshape(-1))


def test_assembly_matches_fancy_index(cfg0):
    c, W, I = cfg0
    o = oracle.evaluate_cached(c, W, I, stages=True)[0]
    H, slot = o["H"], o["slot"]
    gathered = H[slot]                          # [K][L][d]
    pos = W["pos"].astype(np.float64)
    assert np.array_equal(o["seq"][:, 1:], gathered + pos[1:c.L + 1])
    assert np.array_equal(o["seq"][:, 0], np.broadcast_to(W["cls"] + pos[0], (c.K, c.d)))


def test_select_rule():
    rng = np.random.default_rng(4)
    for _ in range(50):
        s = rng.standard_normal(rng.integers(1, 30))
        assert oracle.select(s) == int(np.argmax(s))
    assert oracle.select(np.array([1.0, 3.0, 3.0, 2.0])) == 1            # smallest index among ties
    assert oracle.select(np.array([np.nan, 0.5, np.nan, 0.5])) == 1      # NaN never wins
    assert oracle.select(np.array([np.nan, np.nan])) == -1
    assert oracle.select(np.array([-np.inf, -np.inf])) == 0


# ----------------------------------------------------------------------------- closed forms (P7)

def test_layer_norm_of_constant_row_is_offset():
    g = np.random.default_rng(5).standard_normal(16)
    b = np.random.default_rng(6).standard_normal(16)
    assert np.allclose(oracle.layer_norm(np.full((3, 16), 7.25), g, b), b, atol=0, rtol=0)


def test_layer_norm_known_values():
    x = np.array([[1.0, 2.0, 3.0, 4.0]])
    # mean 2.5, biased variance 1.25
    want = (x - 2.5) / np.sqrt(1.25 + 1e-5)
    assert _rel(oracle.layer_norm(x, np.ones(4), np.zeros(4)), want) < 1e-15


def test_single_key_attention_returns_value():
    rng = np.random.default_rng(7)
    q = rng.standard_normal((5, 8))
    k = rng.standard_normal((1, 8))
    v = rng.standard_normal((1, 8))
    out = oracle.attention(q, k, v, 2)
    assert np.allclose(out, np.broadcast_to(v, (5, 8)), rtol=0, atol=1e-15)


def test_cross_attention_with_one_context_row_ignores_queries():
    """T=1: each item's cross-attention output is (m Wv + bv) Wo2 + bo2 whatever its query."""
    c = gen.config(0, T=1, n_layers=1)
    W = gen.make_weights(c)
    m = np.random.default_rng(8).standard_normal((1, c.d))
    kv = [(m @ W["ctx.kv.0.wk"].astype(np.float64) + W["ctx.kv.0.bk"],
           m @ W["ctx.kv.0.wv"].astype(np.float64) + W["ctx.kv.0.bv"])]
    q = np.random.default_rng(9).standard_normal((4, c.d))
    o = oracle.attention(q, kv[0][0], kv[0][1], c.n_heads)
    want = (m @ W["ctx.kv.0.wv"].astype(np.float64) + W["ctx.kv.0.bv"])
    assert np.allclose(o, np.broadcast_to(want, o.shape), rtol=0, atol=1e-15)


def test_zero_key_projection_gives_mean_of_values():
    rng = np.random.default_rng(10)
    q = rng.standard_normal((3, 12))
    v = rng.standard_normal((9, 12))
    out = oracle.attention(q, np.zeros((9, 12)), v, 3)
    assert np.allclose(out, np.broadcast_to(v.mean(0), out.shape), rtol=0, atol=1e-14)


def test_one_list_cross_sequence_is_value_path():
    """K=1: the cross-sequence attention weight is 1, so each block is x + (LN1(x) Wv + bv) Wo + bo, + FFN."""
    c = gen.config(0, n_layers=1)
    W = gen.make_weights(c)
    x = np.random.default_rng(11).standard_normal((1, c.d))
    d = c.d
    f = lambda a: a.astype(np.float64)
    h = oracle.layer_norm(x, W["cross.0.ln1.g"], W["cross.0.ln1.b"])
    v = h @ f(W["cross.0.wqkv"])[:, 2 * d:] + f(W["cross.0.bqkv"])[2 * d:]
    y = x + v @ f(W["cross.0.wo"]) + f(W["cross.0.bo"])
    h2 = oracle.layer_norm(y, W["cross.0.ln2.g"], W["cross.0.ln2.b"])
    y = y + np.maximum(h2 @ f(W["cross.0.w1"]) + f(W["cross.0.b1"]), 0) @ f(W["cross.0.w2"]) + f(W["cross.0.b2"])
    want = oracle.layer_norm(y, W["cross.lnf.g"], W["cross.lnf.b"])
    assert _rel(oracle.cross_sequence(c, W, x), want) < 1e-14


# ----------------------------------------------------------------------------- invariants (P8-P10, P12)

def _with_lists(I, lists):
    J = dict(I)
    J["lists"] = lists
    return J


def test_scores_permutation_equivariant(cfg1_small):
    c, W, I = cfg1_small
    perm = np.random.default_rng(12).permutation(c.K)
    J = _with_lists(I, I["lists"][:, perm])
    a = oracle.evaluate_cached(c, W, I, requests=[0])[0]
    b = oracle.evaluate_cached(c, W, J, requests=[0])[0]
    assert _rel(b["scores"], a["scores"][perm]) < 1e-12
    assert perm[b["best"]] == a["best"]


def test_without_cross_sequence_lists_are_independent(cfg0):
    """Zeroed cross-sequence output projections and FFN outputs ("-CrossSeq"): s_k depends on list k only."""
    c, W, I = cfg0
    W2 = dict(W)
    for l in range(c.n_layers):
        for n in ("wo", "bo", "w2", "b2"):
            W2[f"cross.{l}.{n}"] = np.zeros_like(W[f"cross.{l}.{n}"])
    a = oracle.evaluate_cached(c, W2, I)[0]["scores"]
    lists = I["lists"].copy()
    lists[0, 2] = (lists[0, 2] + 3) % c.M          # change list 2 only
    b = oracle.evaluate_cached(c, W2, _with_lists(I, lists))[0]["scores"]
    assert a[2] != b[2]
    # item-set attention couples lists through H; a list that keeps its items but whose
    # neighbours change must still be scored identically when U(z) is unchanged.
    lists2 = I["lists"].copy()
    lists2[0, [1, 2]] = lists2[0, [2, 1]]          # swap two lists: same U, same H
    c2 = oracle.evaluate_cached(c, W2, _with_lists(I, lists2))[0]["scores"]
    assert c2[0] == a[0] and c2[3] == a[3]


def test_identical_lists_score_identically(cfg1_small):
    c, W, I = cfg1_small
    lists = np.broadcast_to(I["lists"][:, :1], I["lists"].shape).copy()
    o = oracle.evaluate_cached(c, W, _with_lists(I, lists), requests=[0])[0]
    # equal up to the BLAS reduction order of each row inside a blocked matmul
    s = o["scores"]
    assert np.max(np.abs(s - s[0])) <= 1e-14 * np.max(np.abs(s))
    assert s[o["best"]] == np.max(s)


def test_positions_added_after_gather():
    c = gen.config(0, K=2, L=4)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    lists = np.array([[[3, 7, 3, 1], [7, 3, 1, 3]]], dtype=np.int32)
    o = oracle.evaluate_cached(c, W, _with_lists(I, lists), stages=True)[0]
    pos = W["pos"].astype(np.float64)
    seq = o["seq"]
    # item 3 sits at positions 1 and 3 of list 0 and at position 2 of list 1: one H row serves all
    # three occurrences, and their sequence rows differ exactly by the position rows
    assert o["slot"][0, 0] == o["slot"][0, 2] == o["slot"][1, 1]
    h = o["H"][o["slot"][0, 0]]
    assert np.array_equal(seq[0, 1], h + pos[1])
    assert np.array_equal(seq[0, 3], h + pos[3])
    assert np.array_equal(seq[1, 2], h + pos[2])
    assert np.allclose(seq[0, 1] - seq[0, 3], pos[1] - pos[3], rtol=0, atol=1e-14)
    assert not np.allclose(seq[0, 1], seq[0, 3])


# ----------------------------------------------------------------------------- planted mistakes

@pytest.mark.parametrize("mistake", ["scale_dh", "transpose_wo", "drop_ffn_residual", "head_slice",
                                     "ln_unbiased_var", "pos_before_gather"])
def test_planted_mistakes_are_caught(cfg0, monkeypatch, mistake):
    """Each plausible slip in the oracle, planted on the CPU, breaks agreement with torch or brute force."""
    c, W, I = cfg0
    c = gen.config(0, n_heads=2)
    W = gen.make_weights(c)
    ref = evaluate_torch(c, W, I, 0)["scores"]
    br = oracle.evaluate_brute(c, W, I, 0)["scores"]
    if mistake == "scale_dh":
        monkeypatch.setattr(ev, "attention", lambda q, k, v, nh: _bad_attention(q, k, v, nh, scale_pow=1.0))
    elif mistake == "transpose_wo":
        orig_sab = ev.self_attention_block

        def sab(x, W_, p, nh, kind="softmax"):
            W3 = dict(W_)
            W3[f"{p}.wo"] = np.ascontiguousarray(W_[f"{p}.wo"].T)
            return orig_sab(x, W3, p, nh, kind)
        monkeypatch.setattr(ev, "self_attention_block", sab)
    elif mistake == "drop_ffn_residual":
        def enc(x, W_, p, nh, kind="softmax"):
            x = x + ev.self_attention_block(ev.layer_norm(x, W_[f"{p}.ln1.g"], W_[f"{p}.ln1.b"]), W_, p, nh, kind)
            return ev.ffn(ev.layer_norm(x, W_[f"{p}.ln2.g"], W_[f"{p}.ln2.b"]), W_, p)
        monkeypatch.setattr(ev, "encoder_block", enc)
    elif mistake == "head_slice":
        monkeypatch.setattr(ev, "attention", lambda q, k, v, nh: _bad_attention(q, k, v, nh, swap_heads=True))
    elif mistake == "ln_unbiased_var":
        def ln(x, g, b):
            mu = x.mean(axis=-1, keepdims=True)
            var = ((x - mu) ** 2).sum(axis=-1, keepdims=True) / (x.shape[-1] - 1)
            return np.asarray(g, np.float64) * (x - mu) / np.sqrt(var + ev.LN_EPS) + np.asarray(b, np.float64)
        monkeypatch.setattr(ev, "layer_norm", ln)
    elif mistake == "pos_before_gather":
        def asm(W_, rows):
            return ev.__dict__["_orig_assemble"](W_, rows + np.asarray(W_["pos"], np.float64)[:rows.shape[0]])
        ev.__dict__["_orig_assemble"] = ev.assemble_one
        monkeypatch.setattr(ev, "assemble_one", asm)
    bad = ev.evaluate_cached(c, W, I)[0]["scores"]
    assert _rel(bad, ref) > 1e-6 and _rel(bad, br) > 1e-6


def _bad_attention(q, k, v, n_heads, scale_pow=0.5, swap_heads=False):
    d = q.shape[-1]
    dh = d // n_heads
    out = np.empty((q.shape[0], d))
    for h in range(n_heads):
        cols = slice(h * dh, (h + 1) * dh)
        kc = slice(((h + 1) % n_heads) * dh, ((h + 1) % n_heads + 1) * dh) if swap_heads else cols
        a = ev.softmax_rows(q[:, cols] @ k[:, kc].T / dh ** scale_pow)
        out[:, cols] = a @ v[:, cols]
    return out


def test_golden_reuse_example():
    """Hand-worked instance: U(z), occurrence ranks and the reuse factor."""
    import json
    import os
    with open(os.path.join(os.path.dirname(__file__), "golden", "reuse_example.json")) as f:
        g = json.load(f)
    lists = np.array(g["lists"], dtype=np.int32)
    uniq, slot = oracle.distinct_items(lists)
    assert uniq.tolist() == g["uniq"]
    assert slot.tolist() == g["slot"]
    assert len(uniq) == g["U"]
    assert lists.size / len(uniq) == g["rho"]


# ----------------------------------------------------------- head-side variants (Section 4.4)

def test_without_cross_sequence_variant_matches_torch(cfg1_small):
    """The "- CrossSeq" variant (C' = c) against the pass rebuilt from torch layers without the
    cross-sequence module, and the naive order against the cached one."""
    c, W, I = cfg1_small
    o = oracle.evaluate_cached(c, W, I, requests=[0], cross_seq=False)[0]
    t = evaluate_torch(c, W, I, 0, cross_seq=False)
    assert _rel(o["Cp"], t["Cp"]) < 1e-12
    assert _rel(o["scores"], t["scores"]) < 1e-12
    n = oracle.evaluate_naive(c, W, I, requests=[0], cross_seq=False)[0]
    assert _rel(n["scores"], o["scores"]) < 1e-12
    full = oracle.evaluate_cached(c, W, I, requests=[0])[0]
    assert np.array_equal(o["Cp"], full["c"])          # C' is SeqEnc's output, untouched
    assert not np.allclose(o["scores"], full["scores"])  # and the interaction does change scores


def test_without_cross_sequence_variant_scores_lists_independently(cfg1_small):
    """Without the interaction, a list whose items and U(z) stay the same keeps its score bit for
    bit while the other lists are reordered or replaced by other lists over the same items."""
    c, W, I = cfg1_small
    a = oracle.evaluate_cached(c, W, I, requests=[0], cross_seq=False)[0]["scores"]
    lists = I["lists"].copy()
    lists[0, [1, 2, 3]] = lists[0, [3, 1, 2]]
    b = oracle.evaluate_cached(c, W, _with_lists(I, lists), requests=[0], cross_seq=False)[0]["scores"]
    assert b[0] == a[0] and b[4] == a[4] and b[5] == a[5]
    assert b[1] == a[3] and b[2] == a[1] and b[3] == a[2]


def _objective_heads(d, n_obj, seed=7):
    rng = np.random.default_rng(seed)
    return rng.normal(0, 0.05, (n_obj, d)), rng.normal(0, 0.05, n_obj), rng.uniform(-1, 1, n_obj)


def test_multi_objective_head_reduces_to_single_head(cfg0):
    """One task head with fusion weight 1 is the model's own linear head."""
    c, W, I = cfg0
    Cp = oracle.evaluate_cached(c, W, I)[0]["Cp"]
    obj, fused = oracle.score_objectives(Cp, W["head.w"][None], W["head.b"], np.ones(1))
    ref = oracle.score(W, Cp)
    assert _rel(obj[:, 0], ref) < 1e-12 and _rel(fused, ref) < 1e-12


def test_multi_objective_head_brute_force_and_linearity(cfg0):
    """Per-task scores by scalar loops; the fused score of linear heads is the single linear head
    with w = sum_t alpha_t w_t and b = sum_t alpha_t b_t."""
    c, W, I = cfg0
    Cp = oracle.evaluate_cached(c, W, I)[0]["Cp"]
    hw, hb, al = _objective_heads(c.d, 3)
    obj, fused = oracle.score_objectives(Cp, hw, hb, al)
    for k in range(Cp.shape[0]):
        f = 0.0
        for t in range(3):
            s = sum(float(Cp[k, i]) * float(hw[t, i]) for i in range(c.d)) + float(hb[t])
            assert abs(obj[k, t] - s) <= 1e-12 * (1 + abs(s))
            f += float(al[t]) * s
        assert abs(fused[k] - f) <= 1e-12 * (1 + abs(f))
    w_eq, b_eq = al @ hw, al @ hb
    assert _rel(fused, Cp @ w_eq + b_eq) < 1e-12
    assert oracle.select(fused) == int(np.argmax(fused))
