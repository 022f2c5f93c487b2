"""Seeded workload generator: determinism, sampling rules, bf16 rounding (no GPU)."""
import numpy as np
import pytest
import torch

import gen


def test_same_seed_same_arrays():
    for cid in (0, 1):
        c = gen.config(cid)
        a, b = gen.make_inputs(c), gen.make_inputs(c)
        for k in a:
            if a[k] is not None:
                assert np.array_equal(a[k], b[k])
        wa, wb = gen.make_weights(c), gen.make_weights(c)
        assert all(np.array_equal(wa[k], wb[k]) for k in wa)


def test_param_spec_matches_weights():
    for cid in (0, 1, 3):
        c = gen.config(cid)
        W = gen.make_weights(c)
        spec = gen.param_spec(c)
        assert [n for n, _, _ in spec] == list(W)
        for n, shape, _ in spec:
            assert W[n].shape == shape and W[n].dtype == np.float32


@pytest.mark.parametrize("cid", [1, 3])
def test_no_repeats_within_a_list(cid):
    c = gen.config(cid)
    lists = gen.make_inputs(c)["lists"]
    assert lists.shape == (c.B, c.K, c.L)
    assert lists.min() >= 0 and lists.max() < c.M
    for b in range(c.B):
        for k in range(c.K):
            assert len(set(lists[b, k].tolist())) == c.L


def test_zipf_rank_frequencies():
    """First-draw rank frequencies follow p_r ~ r^-s (chi-square over the top ranks)."""
    rng = np.random.default_rng(0)
    M, s, n = 200, 1.1, 20000
    p = np.arange(1, M + 1, dtype=np.float64) ** -s
    p /= p.sum()
    draws = np.array([rng.choice(M, 1, replace=False, p=p)[0] for _ in range(n)])
    top = 20
    obs = np.bincount(draws, minlength=M)[:top]
    exp = p[:top] * n
    chi2 = float(((obs - exp) ** 2 / exp).sum())
    assert chi2 < 45.3       # 99.9th percentile of chi-square with 20 degrees of freedom


def test_workload1_distinct_counts():
    c = gen.config(1)
    lists = gen.make_inputs(c)["lists"]
    U = np.array([len(np.unique(lists[b])) for b in range(c.B)])
    assert 110 <= U.mean() <= 150
    assert (U <= c.U_cap).all()


def test_text_resample_rate():
    c = gen.config(4)
    lists = gen.make_inputs(c)["lists"]
    # hypotheses of one request share a base sequence; a position differs from the column
    # majority about 20% of the time
    diffs = []
    for b in range(c.B):
        for j in range(c.L):
            col = lists[b, :, j]
            vals, cnt = np.unique(col, return_counts=True)
            diffs.append(1.0 - cnt.max() / c.K)
    assert 0.15 < float(np.mean(diffs)) < 0.25


def test_bf16_rounding_matches_torch():
    x = np.random.default_rng(1).standard_normal(100_000).astype(np.float32) * 3
    x[:4] = [1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -0.0, 65504.0]   # ties to even both ways
    ours = gen.round_bf16(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(ours.view(np.uint32), ref.view(np.uint32))


def test_bf16_workloads_are_bf16_representable():
    c = gen.config(1)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    for a in list(W.values())[:8] + [I["x"], I["pool"]]:
        assert np.array_equal(gen.round_bf16(a), a)


def test_sinusoid_position_table():
    c = gen.config(4)
    pos = gen.make_weights(c)["pos"].astype(np.float64)
    assert pos.shape == (c.L + 1, c.d)
    assert np.array_equal(pos[0, 0::2], np.zeros(c.d // 2))
    assert np.array_equal(pos[0, 1::2], np.ones(c.d // 2))
    # sin^2 + cos^2 = 1 per frequency, up to bf16 rounding of each entry
    assert np.allclose(pos[:, 0::2] ** 2 + pos[:, 1::2] ** 2, 1.0, atol=2 * 2 ** -8)
    assert abs(pos[1, 0] - np.sin(1.0)) < 2 ** -8
