"""Parity of the linear-attention variant (Appendix B.3's deployment setting) of the HIP path with
the float64 oracle: the context's per-head linear-attention state (the variant's key/value
cache), the item encodings, the sequences, C' and the scores/selection."""
import numpy as np
import pytest

import gen
import oracle
from paper_2603_02565_amd import flasheval as fe
from tests.gpu_harness import check_scores, make_evaluator, normwise, rtol_for, run_pass, score_tol, upload

pytestmark = pytest.mark.gpu


def _lin(cid, **kw):
    c = gen.config(cid, attention="linear", **kw)
    return c, gen.make_weights(c), gen.make_inputs(c)


def _amplify(W, n_layers, factor=32.0, qk=4.0):
    """Weights under which the attentions dominate their blocks: output projections of every
    attention scaled by `factor` and the q|k|v projections by `qk` (powers of two, so bf16
    values stay exact).  With N(0, 0.02) weights every attention is near uniform and contributes
    little, so this is where a wrong weight formula would show."""
    W = dict(W)
    for l in range(n_layers):
        for p in (f"ctx.{l}", f"cross.{l}", f"seq.{l}", f"item.{l}"):
            W[f"{p}.wo"] = W[f"{p}.wo"] * factor
            W[f"{p}.wqkv"] = W[f"{p}.wqkv"] * qk
        W[f"item.{l}.wo2"] = W[f"item.{l}.wo2"] * factor
        W[f"item.{l}.wq"] = W[f"item.{l}.wq"] * qk
        W[f"ctx.kv.{l}.wk"] = W[f"ctx.kv.{l}.wk"] * qk
    return W


def _check(c, W, I, out, requests, stages=True):
    tol = rtol_for(c)
    ref = oracle.evaluate_cached(c, W, I, requests=requests, stages=stages)
    for b in requests:
        r = ref[b]
        if stages:
            for l in range(c.n_layers):
                st = oracle.linear_kv_state(r["kv"][l][0], r["kv"][l][1], c.n_heads)
                assert normwise(out["kv"][l, b], st) <= tol, ("linear state", l, b)
            U = len(r["uniq"])
            assert out["n_uniq"][b] == U
            assert np.array_equal(out["uniq"][b, :U], r["uniq"])
            assert np.array_equal(out["slot"][b], r["slot"])
            assert normwise(out["H"][b, :U], r["H"]) <= tol, ("H", b)
            assert normwise(out["seq"][b], r["seq"]) <= tol, ("seq", b)
        assert normwise(out["Cp"][b], r["Cp"]) <= tol, ("Cp", b)
        check_scores(c, out["scores"][b], out["best"][b], r["scores"], b)


def test_state_layout_and_size():
    c, W, I = _lin(1, B=2, K=3, T=40)
    ev = make_evaluator(c, W)
    assert fe.fe_kv_size(ev.handle, 2, 40) == c.n_layers * 2 * c.n_heads * (c.dh + 1) * c.dh * 4
    b = ev.allocate(2, 40, c.M, 3, c.L)
    assert tuple(b["kv"].shape) == (c.n_layers, 2, c.n_heads, c.dh + 1, c.dh)
    ev.close()


def test_linear_cfg0_fp32_matches_naive_oracle():
    c, W, I = _lin(0)
    out = run_pass(c, W, I)
    ref = oracle.evaluate_naive(c, W, I)[0]
    check_scores(c, out["scores"][0], out["best"][0], ref["scores"], "naive")
    _check(c, W, I, out, [0])


def test_linear_cfg0_fp32_amplified():
    c, W, I = _lin(0, n_heads=1, n_layers=2)
    W = _amplify(W, c.n_layers)
    out = run_pass(c, W, I)
    _check(c, W, I, out, [0])


@pytest.mark.parametrize("shape", [dict(B=3, K=7), dict(B=2, K=9, T=37, M=23, L=6)])
def test_linear_bf16_recsys_shapes(shape):
    c, W, I = _lin(1, **shape)
    out = run_pass(c, W, I)
    _check(c, W, I, out, list(range(c.B)))


def test_linear_bf16_amplified():
    c, W, I = _lin(1, B=2, K=6, T=96)
    W = _amplify(W, c.n_layers)
    out = run_pass(c, W, I)
    _check(c, W, I, out, [0, 1])
    # the check discriminates: the softmax network's C' lies well outside the tolerance
    soft = oracle.evaluate_cached(gen.config(1, B=2, K=6, T=96), W, I, requests=[0])[0]
    assert normwise(out["Cp"][0], soft["Cp"]) > 2 * rtol_for(c)


def test_linear_long_context():
    """T = 2048 context rows (d = 256, 8 heads): the state sums 2048 keys per head."""
    c, W, I = _lin(3, B=1, K=5)
    out = run_pass(c, W, I)
    _check(c, W, I, out, [0])


def test_linear_head_width_64_token_ids():
    c, W, I = _lin(4, B=1, T=96, K=3, L=8, n_layers=2)
    out = run_pass(c, W, I)
    _check(c, W, I, out, [0])


def test_linear_wide_cross_set():
    """K = 200 lists: the cross-sequence state sums 200 list vectors per head."""
    c, W, I = _lin(2, K=200, B=2)
    out = run_pass(c, W, I)
    _check(c, W, I, out, [1], stages=False)


def test_linear_permuting_lists_permutes_scores():
    c, W, I = _lin(1, B=2, K=8)
    W = _amplify(W, c.n_layers)
    a = run_pass(c, W, I)
    perm = np.random.default_rng(5).permutation(c.K)
    J = dict(I)
    J["lists"] = np.ascontiguousarray(I["lists"][:, perm])
    b = run_pass(c, W, J)
    ref = oracle.evaluate_cached(c, W, I, requests=[0])[0]
    assert np.max(np.abs(b["scores"][0] - a["scores"][0][perm])) <= score_tol(c, ref["scores"])


def test_linear_naive_evaluator_matches_joint_pass():
    import torch
    c, W, I = _lin(1, B=2, K=4, T=64)
    ev = make_evaluator(c, W)
    B, K, L = I["lists"].shape
    ev.allocate(B, c.T, c.M, K, L)
    d = upload(c, I)
    joint = ev.run(x=d["x"], pool=d["pool"], lists=d["lists"])
    ev.allocate_naive(B, c.T, c.M, K, L, token_ids=False)
    naive = ev.run_naive(x=d["x"], pool=d["pool"], lists=d["lists"])
    torch.cuda.synchronize()
    ref = oracle.evaluate_naive(c, W, I)
    for b in range(B):
        check_scores(c, naive["scores"][b].cpu().numpy(), int(naive["best"][b]), ref[b]["scores"], ("naive", b))
        check_scores(c, joint["scores"][b].cpu().numpy(), int(joint["best"][b]), ref[b]["scores"], ("joint", b))
    ev.close()
