"""Head-side variants of Section 4.4 through the C ABI: the pass without cross-sequence
interaction (fe_encode_sequences, the "- CrossSeq" ablation) and multi-objective heads with a
weighted-sum fusion (fe_score_objectives), against the float64 oracle."""
import numpy as np
import pytest
import torch

import gen
import oracle
from paper_2603_02565_amd import flasheval as fe
from tests.gpu_harness import check_scores, check_selection, make_evaluator, normwise, rtol_for, upload

pytestmark = pytest.mark.gpu


def _act(c):
    return torch.bfloat16 if c.dtype == "bf16" else torch.float32


@pytest.mark.parametrize("cid,shape", [(1, dict(B=3, K=7)), (0, {}), (4, dict(B=1, T=64, K=3, L=8))])
def test_pass_without_cross_sequence(cid, shape):
    """Joint pass with C' = c: context, items and assembly as usual, then SeqEnc alone and the head.
    Workload 4 (d = 512) takes the separate-kernel SeqEnc path, the others the module kernel."""
    c = gen.config(cid, **shape)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    ev = make_evaluator(c, W)
    B, K, L = I["lists"].shape
    T = (I["x"] if I.get("x") is not None else I["ctx_ids"]).shape[1]
    bufs = ev.allocate(B, T, c.M, K, L)
    d = upload(c, I)
    h = ev.handle
    fe.fe_encode_context(h, B, T, d["x"], d["ctx_ids"], bufs["kv"], bufs["ws"])
    fe.fe_encode_items(h, B, c.M, d["pool"], d["lists"], K, L, bufs["kv"], T, bufs["uniq"], bufs["n_uniq"],
                       bufs["slot"], bufs["H"], bufs["ws"])
    fe.fe_assemble(h, B, K, L, bufs["U_cap"], bufs["slot"], bufs["H"], bufs["seq"])
    C = torch.empty((B, K, c.d), dtype=torch.float32, device="cuda")
    fe.fe_encode_sequences(h, B, K, L, bufs["seq"], C, bufs["ws"])
    fe.fe_score_select(h, B, K, C, bufs["scores"], bufs["best"])
    torch.cuda.synchronize()
    Cg, s, best = C.cpu().numpy(), bufs["scores"].cpu().numpy(), bufs["best"].cpu().numpy()
    ref = oracle.evaluate_cached(c, W, I, cross_seq=False)
    tol = rtol_for(c)
    for b in range(B):
        assert normwise(Cg[b], ref[b]["Cp"]) <= tol
        check_scores(c, s[b], best[b], ref[b]["scores"], b)
    ev.close()


def test_encode_sequences_on_oracle_sequences():
    """Stage-isolated: SeqEnc alone on the oracle's assembled sequences (rounded to bf16)."""
    c = gen.config(1, B=2, K=9, L=10)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    ev = make_evaluator(c, W)
    bufs = ev.allocate(c.B, c.T, c.M, c.K, c.L)
    refs = oracle.evaluate_cached(c, W, I, stages=True, cross_seq=False)
    seq = np.stack([refs[b]["seq"] for b in range(c.B)]).astype(np.float32)
    seq_t = torch.from_numpy(seq).cuda().to(torch.bfloat16)
    seq64 = seq_t.float().cpu().numpy().astype(np.float64)
    C = torch.empty((c.B, c.K, c.d), dtype=torch.float32, device="cuda")
    fe.fe_encode_sequences(ev.handle, c.B, c.K, c.L, seq_t, C, bufs["ws"])
    Cg = C.cpu().numpy()
    for b in range(c.B):
        want = np.stack([oracle.encode_sequence(c, W, seq64[b, k]) for k in range(c.K)])
        assert normwise(Cg[b], want) <= rtol_for(c)
    ev.close()


def _heads(d, n_obj, seed=11):
    rng = np.random.default_rng(seed)
    return (rng.normal(0, 0.05, (n_obj, d)).astype(np.float32), rng.normal(0, 0.05, n_obj).astype(np.float32),
            rng.uniform(-1, 1, n_obj).astype(np.float32))


@pytest.mark.parametrize("cid,d,n_obj", [(1, 128, 3), (0, 32, 1), (1, 512, 8)])
def test_score_objectives_on_oracle_inputs(cid, d, n_obj):
    c = gen.config(cid, B=3, K=50, d=d, n_heads=d // 32 if d <= 128 else d // 64, ffn=4 * d)
    W = gen.make_weights(c)
    ev = make_evaluator(c, W)
    rng = np.random.default_rng(3)
    Cp = rng.standard_normal((c.B, c.K, d)).astype(np.float32)
    Cp[1, 9] = Cp[1, 4]                        # tie between lists 4 and 9
    Cp[2, 30:] = np.nan                        # NaN lists never win
    hw, hb, al = _heads(d, n_obj)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    obj = torch.empty((c.B, c.K, n_obj), dtype=torch.float32, device="cuda")
    fused = torch.empty((c.B, c.K), dtype=torch.float32, device="cuda")
    best = torch.empty((c.B,), dtype=torch.int32, device="cuda")
    fe.fe_score_objectives(ev.handle, c.B, c.K, dev(Cp), n_obj, dev(hw), dev(hb), dev(al), obj, fused, best)
    torch.cuda.synchronize()
    og, fg, bg = obj.cpu().numpy(), fused.cpu().numpy(), best.cpu().numpy()
    eps = 2.0 ** -24
    for b in range(c.B):
        o_ref, f_ref = oracle.score_objectives(Cp[b].astype(np.float64), hw, hb, al)
        ok = ~np.isnan(f_ref)
        assert np.array_equal(np.isnan(fg[b]), ~ok)
        # forward-error bound of a d-term fp32 dot product, then of the n_obj-term fusion
        term = np.abs(Cp[b][ok].astype(np.float64)) @ np.abs(hw.astype(np.float64)).T + np.abs(hb)
        assert np.all(np.abs(og[b][ok] - o_ref[ok]) <= (d + 2) * eps * term)
        fbound = (d + n_obj + 2) * eps * (term @ np.abs(al.astype(np.float64)))
        assert np.all(np.abs(fg[b][ok] - f_ref[ok]) <= fbound)
        # selection on the fused scores the kernel produced: exact tie and NaN rules
        assert bg[b] == oracle.select(fg[b].astype(np.float64))
        check_selection(int(bg[b]), np.where(ok, f_ref, -np.inf), float(fbound.max()))
    with pytest.raises(fe.FeError) as e:
        fe.fe_score_objectives(ev.handle, c.B, c.K, dev(Cp), 9, dev(np.zeros((9, d), np.float32)), dev(hb),
                               dev(al), obj, fused, best)
    assert e.value.status == fe.FE_EUNSUPPORTED
    ev.close()
