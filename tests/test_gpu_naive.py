"""The candidate-factorised evaluator on the GPU (fe_evaluate_naive): the same network with every
reuse taken out.  Its results must equal the oracle's candidate-factorised evaluation and the
joint pass's (QKV-Cache reuses exact results, Section 4.2)."""
import numpy as np
import pytest
import torch

import gen
import oracle
from tests.gpu_harness import check_scores, make_evaluator, normwise, rtol_for, run_pass, upload

pytestmark = pytest.mark.gpu


def _run_naive(c, W, I, ev=None):
    own = ev is None
    if own:
        ev = make_evaluator(c, W)
    B, K, L = I["lists"].shape
    T = (I["x"] if I.get("x") is not None else I["ctx_ids"]).shape[1]
    ev.allocate_naive(B, T, c.M, K, L, token_ids=I.get("ctx_ids") is not None)
    d = upload(c, I)
    b = ev.run_naive(x=d["x"], ctx_ids=d["ctx_ids"], pool=d["pool"], lists=d["lists"])
    torch.cuda.synchronize()
    out = {k: b[k].cpu().numpy() for k in ("Cp", "scores", "best")}
    if own:
        ev.close()
    return out


def _check_against(c, W, got, ref_scores, ref_Cp, b):
    tol = rtol_for(c)
    assert normwise(got["Cp"][b], ref_Cp) <= tol, "Cp"
    check_scores(c, got["scores"][b], got["best"][b], ref_scores, b)


def test_naive_cfg0_fp32_matches_oracle_naive():
    c = gen.config(0)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    got = _run_naive(c, W, I)
    ref = oracle.evaluate_naive(c, W, I)[0]
    _check_against(c, W, got, ref["scores"], ref["Cp"], 0)


@pytest.mark.parametrize("shape", [dict(B=2, K=6, L=5), dict(B=2, T=37, M=23, K=9, L=6)])
def test_naive_bf16_matches_oracle_and_joint(shape):
    c = gen.config(1, **shape)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    got = _run_naive(c, W, I)
    joint = run_pass(c, W, I)
    naive0 = oracle.evaluate_naive(c, W, I, requests=[0])[0]
    _check_against(c, W, got, naive0["scores"], naive0["Cp"], 0)
    cached = oracle.evaluate_cached(c, W, I)
    for b in range(c.B):
        _check_against(c, W, got, cached[b]["scores"], cached[b]["Cp"], b)
        # same kernels on identical encodings: the joint pass's results to rounding order
        assert normwise(got["Cp"][b], joint["Cp"][b]) <= rtol_for(c)


def test_naive_text_hypotheses_token_ids():
    c = gen.config(4, B=1, T=128, K=3, L=8)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    got = _run_naive(c, W, I)
    ref = oracle.evaluate_cached(c, W, I)[0]
    _check_against(c, W, got, ref["scores"], ref["Cp"], 0)


def test_naive_rejects_bad_arguments():
    from paper_2603_02565_amd import flasheval as fe
    c = gen.config(1, B=1, K=2, L=3)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    ev = make_evaluator(c, W)
    ev.allocate_naive(1, c.T, c.M, 2, 3, token_ids=False)
    d = upload(c, I)
    b = ev.naive_buffers
    small = torch.empty(256, dtype=torch.uint8, device=b["ws"].device)
    with pytest.raises(fe.FeError) as e:
        fe.fe_evaluate_naive(ev.handle, 1, c.T, c.M, 2, 3, d["x"], None, d["pool"], d["lists"], b["Cp"], b["scores"],
                             b["best"], small)
    assert e.value.status == fe.FE_EINVAL
    with pytest.raises(fe.FeError) as e:   # neither x nor ctx_ids
        fe.fe_evaluate_naive(ev.handle, 1, c.T, c.M, 2, 3, None, None, d["pool"], d["lists"], b["Cp"], b["scores"],
                             b["best"], b["ws"])
    assert e.value.status == fe.FE_EINVAL
    ev.close()
