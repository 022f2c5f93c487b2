"""The bench's algorithmic flop accounting: however the pass's flops are split over kernel
families, they add up to the per-stage totals of the joint pass (Section 5.2, Appendix A.3 cost
model; the last sequence-encoder block computes keys and values for every row but the rest only
for the [CLS] rows)."""
import pytest

import bench
import gen


def _block(d, F, rows, groups, size):
    """One pre-LN encoder block: q|k|v and output projections, FFN, attention inside groups."""
    return rows * (8.0 * d * d + 4.0 * d * F) + groups * 4.0 * size * size * d


def _joint_total(c, U):
    d, F, n, B, T, K, S = c.d, c.ffn, c.n_layers, c.B, c.T, c.K, c.L + 1
    ctx = n * _block(d, F, B * T, B, T)
    kv = 4.0 * n * B * T * d * d
    items = sum(n * (u * (12.0 * d * d + 4.0 * d * F) + 4.0 * u * u * d + 4.0 * u * T * d) for u in U)
    seq = (n - 1) * _block(d, F, B * K * S, B * K, S)
    seq += B * K * S * 4.0 * d * d + B * K * (4.0 * d * d + 4.0 * d * F + 4.0 * S * d)
    cross = n * _block(d, F, B * K, B, K)
    return ctx + kv + items + seq + cross


@pytest.mark.parametrize("cid,kw", [(1, {}), (2, {"K": 1000}), (3, {}), (4, {}), (0, {})])
def test_family_split_adds_up_to_the_joint_pass(cid, kw):
    c = gen.config(cid, **kw)
    U = [min(c.M, c.K * c.L) - 3] * c.B
    fams = {"layer", "post", "attention", "gemm"}
    split = bench.family_flops(c, U, fams)
    assert set(split) <= fams | {"linear"}
    assert sum(split.values()) == pytest.approx(_joint_total(c, U), rel=1e-12)


def test_fused_cross_attention_carries_the_item_projections():
    """On the RecSys model the item layers' output and query projections run inside the fused
    cross-attention kernel, so the attention family, not the tail family, carries them."""
    c = gen.config(1)
    U = [129] * c.B
    f = bench.family_flops(c, U, {"layer", "post", "attention", "gemm"})
    d, F, n, T = c.d, c.ffn, c.n_layers, c.T
    rows = sum(U)
    attn = sum(n * (4.0 * u * u * d + 4.0 * u * T * d) for u in U) + n * 6.0 * d * d * rows + n * 4.0 * d * d * rows
    attn += n * 4.0 * c.B * T * T * d + n * 6.0 * d * d * c.B * T           # context self-attention with its q|k|v
    assert f["attention"] == pytest.approx(attn, rel=1e-12)
