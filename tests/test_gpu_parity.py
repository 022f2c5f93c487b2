"""Parity of the HIP path (through the C ABI) with the float64 oracle, stage by stage and end to end."""
import numpy as np
import pytest
import torch

import gen
import oracle
from paper_2603_02565_amd import flasheval as fe
from tests.gpu_harness import check_scores, fetch, make_evaluator, normwise, rtol_for, run_pass, score_tol, upload
from tests.oracle_pool import compare_batch

pytestmark = pytest.mark.gpu


def _stage_refs(cfg, W, I, b):
    return oracle.evaluate_cached(cfg, W, I, requests=[b], stages=True)[b]


def _compare_request(cfg, W, out, ref, b, check_kv=True):
    tol = rtol_for(cfg)
    if check_kv:
        for l in range(cfg.n_layers):
            assert normwise(out["kv"][l, 0, b], ref["kv"][l][0]) <= tol, ("K cache", l)
            assert normwise(out["kv"][l, 1, b], ref["kv"][l][1]) <= tol, ("V cache", l)
    U = len(ref["uniq"])
    assert out["n_uniq"][b] == U
    assert np.array_equal(out["uniq"][b, :U], ref["uniq"])
    assert np.all(out["uniq"][b, U:] == -1)
    assert np.array_equal(out["slot"][b], ref["slot"])
    assert normwise(out["H"][b, :U], ref["H"]) <= tol, "H"
    assert np.all(out["H"][b, U:] == 0)
    assert normwise(out["seq"][b], ref["seq"]) <= tol, "seq"
    assert normwise(out["Cp"][b], ref["Cp"]) <= tol, "Cp"
    if len(ref["scores"]) == 1:
        # one list: a single score, whose size says nothing about its error (its d terms may
        # cancel to almost nothing); it must be the head applied to this C' -- the oracle's score
        # plus the propagated C' error and the fp32 dot product's own rounding -- and be selected
        w = np.abs(W["head.w"].astype(np.float64))
        Cg = out["Cp"][b, 0].astype(np.float64)
        bound = np.abs(Cg - ref["Cp"][0]) @ w + (cfg.d + 2) * 2.0 ** -24 * (np.abs(Cg) @ w + abs(float(W["head.b"][0])))
        assert abs(float(out["scores"][b, 0]) - ref["scores"][0]) <= bound, "scores"
        assert int(out["best"][b]) == 0
        return {"ratio": 0.0, "strict": True}
    return check_scores(cfg, out["scores"][b], out["best"][b], ref["scores"], b)


def check_whole_batch(c, out, requests=None):
    """Every request of a full-size batch (or the listed ones) against the cached-order oracle
    (stage by stage, element by element); prints the measured worst error ratios and the fraction
    of requests in the exact-selection regime."""
    tol = rtol_for(c)
    worst = {k: 0.0 for k in ("kv", "H", "seq", "Cp", "scores")}
    strict = 0
    n = 0
    for r in compare_batch(c, out, requests):
        b, n = r["b"], n + 1
        assert r["n_uniq_ok"] and r["uniq_ok"] and r["slot_ok"], (c.label, b, "distinct set or slots differ")
        assert r["H_pad_zero"], (c.label, b, "padding rows of H are not zero")
        for k in ("H", "seq", "Cp"):
            assert r[k] <= tol, (c.label, b, k, r[k])
            worst[k] = max(worst[k], r[k])
        if "kv" in r:
            assert max(r["kv"]) <= tol, (c.label, b, "kv", r["kv"])
            worst["kv"] = max(worst["kv"], max(r["kv"]))
        m = check_scores(c, out["scores"][b], out["best"][b], r["scores_ref"], (c.label, b))
        worst["scores"] = max(worst["scores"], m["ratio"])
        strict += m["strict"]
    assert np.all(out["status"] == 0)
    print(f"\n[parity] {c.label}: {n} of {c.B} requests; worst normwise error " +
          ", ".join(f"{k} {v:.3g}" for k, v in worst.items()) +
          f"; exact-selection regime {strict}/{n}", flush=True)
    return worst, strict


def test_cfg0_all_stages_fp32():
    c = gen.config(0)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    out = run_pass(c, W, I)
    ref = _stage_refs(c, W, I, 0)
    m = _compare_request(c, W, out, ref, 0)
    assert m["strict"]
    naive = oracle.evaluate_naive(c, W, I)[0]
    check_scores(c, out["scores"][0], out["best"][0], naive["scores"], "naive")
    assert int(out["best"][0]) == naive["best"]
    assert out["status"][0] == 0


@pytest.fixture(scope="module")
def cfg1_out():
    c = gen.config(1)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    return c, W, I, run_pass(c, W, I)


def test_cfg1_every_request(cfg1_out):
    c, W, I, out = cfg1_out
    check_whole_batch(c, out)


def test_cfg1_distinct_sets_all_requests(cfg1_out):
    c, W, I, out = cfg1_out
    for b in range(c.B):
        u, inv = np.unique(I["lists"][b], return_inverse=True)
        assert out["n_uniq"][b] == len(u)
        assert np.array_equal(out["uniq"][b, :len(u)], u)
        assert np.array_equal(out["slot"][b].reshape(-1), inv.reshape(-1))
    assert np.all(out["status"] == 0)


@pytest.mark.parametrize("b", [0, 63])
def test_cfg1_naive_oracle(cfg1_out, b):
    """Requests 0 and B-1 against the candidate-factorised oracle itself (context per list, items
    per occurrence)."""
    c, W, I, out = cfg1_out
    naive = oracle.evaluate_naive(c, W, I, requests=[b])[b]
    assert normwise(out["Cp"][b], naive["Cp"]) <= rtol_for(c)
    check_scores(c, out["scores"][b], out["best"][b], naive["scores"], ("naive", b))


@pytest.mark.parametrize("K", gen.K_SWEEP)
def test_cfg2_k_sweep(K):
    c = gen.config(2, K=K)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    out = run_pass(c, W, I)
    check_whole_batch(c, out)
    if K == 10:
        for b in (0, c.B - 1):
            naive = oracle.evaluate_naive(c, W, I, requests=[b])[b]
            check_scores(c, out["scores"][b], out["best"][b], naive["scores"], ("naive", b))


def test_cfg3_long_context():
    c = gen.config(3)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    out = run_pass(c, W, I)
    check_whole_batch(c, out)


@pytest.mark.parametrize("cid", [1, 3])
def test_linear_attention_every_request(cid):
    """The linear-attention workloads the bench times (RecSys base, long context), every request:
    the per-head state that replaces the key/value cache (its key ranges split over workgroups and
    merged in order), H, the sequences, C', scores and selection."""
    c = gen.config(cid, attention="linear")
    W, I = gen.make_weights(c), gen.make_inputs(c)
    out = run_pass(c, W, I)
    check_whole_batch(c, out)


def test_cfg4_text_hypotheses():
    c = gen.config(4)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    out = run_pass(c, W, I)
    check_whole_batch(c, out)


def test_long_context_ragged_query_groups():
    """Head width 32, 2000 context rows over 128 (request, head) pairs: the chunked attention puts
    eight query tiles on each wave and the last query group of every pair is ragged (first and last
    request)."""
    c = gen.config(3, T=2000)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    out = run_pass(c, W, I)
    check_whole_batch(c, out, requests=[0, c.B - 1])


def test_wide_heads_two_query_tiles_per_wave():
    """Head width 64 with 128 (request, head) pairs of 1024 queries: the chunked attention puts
    two query tiles on each wave (text-hypothesis shapes at 16 requests; first and last request)."""
    c = gen.config(4, B=16)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    out = run_pass(c, W, I)
    check_whole_batch(c, out, requests=[0, c.B - 1])


@pytest.mark.parametrize("cid,B", [(1, 2), (1, 24), (3, 6)])
def test_tails_split_by_hidden_width(cid, B):
    """Tails of launches with few 64-row tiles run as several workgroups per tile, each over a
    slice of the FFN's hidden chunks, with the fp32 partial sums added in a fixed order by a second
    kernel: d = 128 at two requests (context and item tails in four parts), at 24 requests (two
    parts), and d = 256 at six requests (item tails in four parts, cross-sequence tails in eight).
    First and last request against the oracle, stage by stage."""
    c = gen.config(cid, B=B)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    out = run_pass(c, W, I)
    check_whole_batch(c, out, requests=[0, c.B - 1])


# ------------------------------------------------------------------------- stage-isolated parity

@pytest.mark.parametrize("cid,ffn", [(1, 256), (1, 768), (3, 512)])
def test_ffn_width_other_than_4d(cid, ffn):
    """F != 4d: the row-tile tails and module kernels stream the FFN with a runtime chunk count
    (F = 4d takes the compile-time, software-pipelined stream)."""
    kw = dict(B=2, K=20) if cid == 1 else dict(B=1, K=12, T=300, M=120)
    c = gen.config(cid, ffn=ffn, **kw)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    out = run_pass(c, W, I)
    for b in range(c.B):
        _compare_request(c, W, out, _stage_refs(c, W, I, b), b)
    assert np.all(out["status"] == 0)


@pytest.mark.parametrize("d,H,n", [(128, 2, 1), (128, 4, 3), (128, 2, 8), (256, 4, 2), (256, 8, 1)])
def test_model_shapes(d, H, n):
    """Head widths 32 and 64, one to eight layers, d = 128 and 256 on the bf16 path: other kernel
    instantiations (head width 64 takes the chunked attention instead of the fused per-head kernels)."""
    c = gen.config(1, B=2, K=12, L=6, T=80, M=60, d=d, n_heads=H, n_layers=n, ffn=4 * d)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    out = run_pass(c, W, I)
    for b in range(c.B):
        _compare_request(c, W, out, _stage_refs(c, W, I, b), b)


def test_assemble_bit_exact_on_oracle_inputs():
    """fe_assemble on H and slot given by the oracle: the gather is exact; the position add rounds once."""
    c = gen.config(1, B=4)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    ev = make_evaluator(c, W)
    bufs = ev.allocate(c.B, c.T, c.M, c.K, c.L)
    U_cap = bufs["U_cap"]
    H = np.zeros((c.B, U_cap, c.d), np.float32)
    slot = np.zeros((c.B, c.K, c.L), np.int32)
    for b in range(c.B):
        ref = _stage_refs(c, W, I, b)
        H[b, :len(ref["uniq"])] = ref["H"]
        slot[b] = ref["slot"]
    Hb = torch.from_numpy(H).cuda().to(torch.bfloat16)
    sl = torch.from_numpy(slot).cuda()
    fe.fe_assemble(ev.handle, c.B, c.K, c.L, U_cap, sl, Hb, bufs["seq"])
    seq = bufs["seq"].float().cpu().numpy()
    Hr = Hb.float().cpu().numpy().astype(np.float64)
    pos = W["pos"].astype(np.float64)
    want = np.empty_like(seq, dtype=np.float64)
    for b in range(c.B):
        want[b, :, 0] = W["cls"].astype(np.float64) + pos[0]
        want[b, :, 1:] = Hr[b][slot[b]] + pos[1:c.L + 1]
    # one bf16 rounding of an exactly formed fp32 sum
    want_bf16 = torch.from_numpy(want.astype(np.float32)).to(torch.bfloat16).float().numpy()
    assert np.array_equal(seq, want_bf16)
    ev.close()


def test_score_select_on_oracle_inputs():
    c = gen.config(1, B=3)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    ev = make_evaluator(c, W)
    bufs = ev.allocate(c.B, c.T, c.M, c.K, c.L)
    Cp = np.random.default_rng(5).standard_normal((c.B, c.K, c.d)).astype(np.float32)
    Cp[1, 7] = Cp[1, 3]                        # tie between lists 3 and 7
    Cp[2] = Cp[2, 0]                           # every list identical
    Cp[1, 40:] = np.nan                        # NaN scores never win
    Cpt = torch.from_numpy(Cp).cuda()
    fe.fe_score_select(ev.handle, c.B, c.K, Cpt, bufs["scores"], bufs["best"])
    s = bufs["scores"].cpu().numpy()
    best = bufs["best"].cpu().numpy()
    for b in range(c.B):
        ref = oracle.score(W, Cp[b].astype(np.float64))
        ok = ~np.isnan(ref)
        assert np.array_equal(np.isnan(s[b]), ~ok)
        assert normwise(s[b][ok], ref[ok]) <= 1e-5
    assert best[2] == 0
    assert best[1] == oracle.select(s[1].astype(np.float64))
    assert best[0] == oracle.select(s[0].astype(np.float64))
    ev.close()


# ------------------------------------------------------------------------- invariants and edge cases

def test_permuting_lists_permutes_scores():
    c = gen.config(1, B=2)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    ev = make_evaluator(c, W)
    a = run_pass(c, W, I, ev)
    perm = np.random.default_rng(9).permutation(c.K)
    J = dict(I, lists=np.ascontiguousarray(I["lists"][:, perm]))
    p = run_pass(c, W, J, ev)
    ev.close()
    for b in range(c.B):
        # the distinct set and H are unchanged by a list permutation: bitwise
        assert np.array_equal(p["H"][b], a["H"][b])
        assert np.array_equal(p["seq"][b], a["seq"][b][perm])
        assert np.max(np.abs(p["scores"][b] - a["scores"][b][perm])) <= score_tol(c, a["scores"][b])


def test_identical_lists_identical_scores():
    c = gen.config(1, B=2)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    J = dict(I, lists=np.ascontiguousarray(np.broadcast_to(I["lists"][:, :1], I["lists"].shape)))
    out = run_pass(c, W, J)
    for b in range(c.B):
        assert np.all(out["scores"][b] == out["scores"][b][0])
        assert out["best"][b] == 0


def test_two_runs_bitwise_identical():
    c = gen.config(1, B=4)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    ev = make_evaluator(c, W)
    a = run_pass(c, W, I, ev)
    b = run_pass(c, W, I, ev)
    ev.close()
    for k in ("kv", "H", "seq", "Cp", "scores", "best", "slot", "uniq"):
        assert np.array_equal(a[k], b[k]), k


@pytest.mark.parametrize("K,L", [(1, 1), (1, 10), (3, 1), (33, 7)])
def test_small_and_ragged_shapes(K, L):
    c = gen.config(1, B=3, K=K, L=L)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    out = run_pass(c, W, I)
    for b in range(c.B):
        _compare_request(c, W, out, _stage_refs(c, W, I, b), b, check_kv=(b == 0))


def test_ragged_context_and_pool():
    """T and U not multiples of any tile: T=37, M=23 < K*L."""
    c = gen.config(1, B=2, T=37, M=23, K=9, L=6)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    out = run_pass(c, W, I)
    for b in range(c.B):
        _compare_request(c, W, out, _stage_refs(c, W, I, b), b)


def test_bad_index_sets_status_and_zero_row():
    c = gen.config(1, B=2, K=5)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    lists = I["lists"].copy()
    lists[1, 2, 3] = c.M + 5
    lists[1, 4, 0] = -1
    out = run_pass(c, W, dict(I, lists=lists))
    assert out["status"][0] == 0
    assert out["status"][1] & fe.FE_DEV_BAD_INDEX
    assert out["slot"][1, 2, 3] == -1 and out["slot"][1, 4, 0] == -1
    assert np.all(out["seq"][1, 2, 4] == 0) and np.all(out["seq"][1, 4, 1] == 0)


@pytest.mark.parametrize("cid,shape", [
    (0, dict(B=2)),                                    # fp32 model: distinct set and rows in one launch
    (3, dict(B=2, T=64, K=30, L=20)),                  # d = 256, 500 distinct slots: separate set and row gathers
    (4, dict(B=2, T=64, K=3, L=8)),                    # token ids: the set keyed on the vocabulary
])
def test_bad_index_on_separate_set_kernels(cid, shape):
    """List entries outside [0, M) on the kernels that build the distinct set outside the first
    item self-attention: the request's status word gets FE_DEV_BAD_INDEX, the entries' slots are
    -1 and their sequence rows zero; the other request is unaffected and matches the oracle."""
    c = gen.config(cid, **shape)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    lists = I["lists"].copy()
    lists[1, 0, 1] = c.M
    lists[1, c.K - 1, c.L - 1] = -7
    out = run_pass(c, W, dict(I, lists=lists))
    assert out["status"][0] == 0
    assert out["status"][1] == fe.FE_DEV_BAD_INDEX
    assert out["slot"][1, 0, 1] == -1 and out["slot"][1, c.K - 1, c.L - 1] == -1
    assert np.all(out["seq"][1, 0, 2] == 0) and np.all(out["seq"][1, c.K - 1, c.L] == 0)
    _compare_request(c, W, out, _stage_refs(c, W, I, 0), 0)


def test_bad_token_sets_status():
    """Context token ids outside [0, vocab): FE_DEV_BAD_TOKEN in that request's status word only;
    the other request matches the oracle."""
    c = gen.config(4, B=2, T=64, K=3, L=8)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    ids = I["ctx_ids"].copy()
    ids[1, 5] = c.vocab
    ids[1, 63] = -1
    out = run_pass(c, W, dict(I, ctx_ids=ids))
    assert out["status"][0] == 0
    assert out["status"][1] == fe.FE_DEV_BAD_TOKEN
    _compare_request(c, W, out, _stage_refs(c, W, I, 0), 0)


def test_nan_context_selects_minus_one():
    c = gen.config(1, B=2, K=5)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    x = I["x"].copy()
    x[1] = np.nan
    out = run_pass(c, W, dict(I, x=x))
    assert out["best"][1] == -1
    assert out["best"][0] >= 0


def test_host_validation_errors():
    c = gen.config(1, B=2, K=5)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    ev = make_evaluator(c, W)
    bufs = ev.allocate(c.B, c.T, c.M, c.K, c.L)
    d = upload(c, I)
    with pytest.raises(fe.FeError) as e:           # both x and ctx_ids
        fe.fe_encode_context(ev.handle, c.B, c.T, d["x"], d["lists"], bufs["kv"], bufs["ws"])
    assert e.value.status == fe.FE_EINVAL
    small = bufs["ws"][:1024]
    with pytest.raises(fe.FeError) as e:           # workspace too small
        fe.fe_encode_context(ev.handle, c.B, c.T, d["x"], None, bufs["kv"], small)
    assert e.value.status == fe.FE_EINVAL
    with pytest.raises(fe.FeError) as e:           # L beyond the position table
        fe.fe_assemble(ev.handle, c.B, c.K, c.max_L + 1, bufs["U_cap"], bufs["slot"], bufs["H"], bufs["seq"])
    assert e.value.status == fe.FE_EINVAL
    with pytest.raises(fe.FeError) as e:           # misaligned pointer
        fe.fe_assemble(ev.handle, c.B, c.K, c.L, bufs["U_cap"], bufs["slot"].data_ptr() + 4, bufs["H"], bufs["seq"])
    assert e.value.status == fe.FE_EINVAL
    with pytest.raises(fe.FeError) as e:
        fe.fe_workspace_size(ev.handle, c.B, 9000, c.M, c.K, c.L)
    assert e.value.status == fe.FE_EUNSUPPORTED
    ev.close()


def test_graph_replay_matches_eager():
    """The five calls captured as one HIP graph: every replay reproduces the eager pass bit for bit,
    with eager passes on other inputs and cleared outputs between the replays."""
    c = gen.config(1, B=4)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    ev = make_evaluator(c, W)
    B, K, L = I["lists"].shape
    ev.allocate(B, c.T, c.M, K, L)
    d = upload(c, I)
    eager = fetch(ev.run(x=d["x"], pool=d["pool"], lists=d["lists"]))
    other = torch.flip(d["lists"], dims=[1]).contiguous()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        ev.run(x=d["x"], pool=d["pool"], lists=d["lists"])
    torch.cuda.synchronize()
    for _ in range(3):
        ev.run(x=d["x"], pool=d["pool"], lists=other)          # eager work on other inputs
        torch.cuda.synchronize()
        for k in ("kv", "H", "seq", "Cp", "scores"):
            ev.buffers[k].fill_(-7.0)
        for k in ("uniq", "n_uniq", "slot", "best"):
            ev.buffers[k].fill_(-7)
        torch.cuda.synchronize()
        graph.replay()
        got = fetch(ev.buffers)
        for k in ("kv", "uniq", "n_uniq", "slot", "H", "seq", "Cp", "scores", "best"):
            assert np.array_equal(got[k], eager[k]), k
    del graph
    ev.close()


def test_trace_launch_records_match_family_totals():
    """Per-launch trace records (what the bench uses to find the longest kernel of the pass) agree
    with the per-family totals, and the pass ends with assembly, the sequence-encoder module, the
    cross-sequence module and the head."""
    from collections import Counter
    c = gen.config(1, B=2, K=8)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    ev = make_evaluator(c, W)
    ev.allocate(c.B, c.T, c.M, c.K, c.L)
    d = upload(c, I)

    def run():
        ev.run(x=d["x"], pool=d["pool"], lists=d["lists"])
        torch.cuda.synchronize()

    run()
    fe.fe_trace_enable(True)
    run()
    seq = fe.fe_trace_read_launches()
    run()
    tot = fe.fe_trace_read()
    fe.fe_trace_enable(False)
    counts = Counter(f for f, _ in seq)
    assert all(tot[f][1] == counts.get(f, 0) for f in tot)
    assert all(t > 0 for _, t in seq)
    fams = [f for f, _ in seq]
    a = len(fams) - 1 - fams[::-1].index("assemble")
    assert fams[a + 1:] == ["layer", "layer", "score_select"]
    ev.close()
