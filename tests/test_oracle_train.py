"""Pins of the float64 training reference (Section 4.5, Appendix B.1): its forward equals the
numpy oracle's, its gradients equal central finite differences of the loss, the losses reduce to
their closed forms, and the labels follow the min-argmax rule."""
import math

import numpy as np
import pytest
import torch

import gen
import oracle
from oracle import train



@pytest.fixture(autouse=True)
def _float64_default():
    """float64 as torch's default dtype inside these tests only (restored afterwards, so other test
    modules collected in the same process keep float32)."""
    old = torch.get_default_dtype()
    torch.set_default_dtype(torch.float64)
    yield
    torch.set_default_dtype(old)


def _tiny(cid=0, **kw):
    c = gen.config(cid, **kw)
    return c, gen.make_weights(c), gen.make_inputs(c)


@pytest.mark.parametrize("cid,kw", [(0, {}), (1, dict(B=2, K=5, L=4, T=12, M=15, n_layers=1)),
                                    (4, dict(B=1, K=3, L=5, T=9, vocab=40, n_layers=1, d=64, n_heads=1, ffn=128))])
def test_forward_equals_numpy_oracle(cid, kw):
    c, W, I = _tiny(cid, **kw)
    P = {k: torch.tensor(np.asarray(v, np.float64)) for k, v in W.items()}
    for b in range(c.B):
        s = train.request_scores(c, P, I, b).numpy()
        ref = oracle.evaluate_cached(c, W, I, requests=[b])[b]["scores"]
        assert np.max(np.abs(s - ref)) <= 1e-12 * max(1.0, np.max(np.abs(ref)))


def _loss_of(c, W, I, a, kind):
    return train.train_grads(c, W, I, a, kind)[0]


@pytest.mark.parametrize("kind", train.LOSSES)
def test_gradients_equal_finite_differences(kind):
    c, W, I = _tiny(0, K=4, L=3, T=6, M=9)
    W = {k: np.asarray(v, np.float64) for k, v in W.items()}
    a = gen.make_relevance(c)
    a[0, :3] = 1                                       # some positives, so the labels are not all ties
    _, g, _ = train.train_grads(c, W, I, a, kind)
    rng = np.random.default_rng(1)
    names = ["ctx.0.wqkv", "ctx.0.ln1.g", "ctx.lnf.b", "ctx.kv.0.wk", "ctx.kv.0.bv", "item.0.wqkv", "item.0.wq",
             "item.0.wo2", "item.0.ln3.g", "item.0.w1", "item.lnf.g", "seq.0.wo", "seq.0.b2", "seq.lnf.g",
             "cross.0.wqkv", "cross.0.w2", "cross.lnf.b", "cls", "pos", "head.w", "head.b"]
    for name in names:
        for _ in range(2):
            idx = tuple(int(rng.integers(0, n)) for n in W[name].shape)
            h = 1e-6 * max(1.0, abs(W[name][idx]))
            Wp = dict(W); Wp[name] = W[name].copy(); Wp[name][idx] += h
            Wm = dict(W); Wm[name] = W[name].copy(); Wm[name][idx] -= h
            fd = (_loss_of(c, Wp, I, a, kind) - _loss_of(c, Wm, I, a, kind)) / (2 * h)
            assert abs(fd - g[name][idx]) <= 1e-6 * max(1e-3, abs(fd)), (name, idx, fd, g[name][idx])


def test_token_embedding_gradient_equals_finite_difference():
    c, W, I = _tiny(4, B=1, K=3, L=4, T=6, vocab=25, n_layers=1, d=64, n_heads=1, ffn=128)
    W = {k: np.asarray(v, np.float64) for k, v in W.items()}
    a = gen.make_relevance(c)
    _, g, _ = train.train_grads(c, W, I, a, "ce")
    for e in (int(I["ctx_ids"][0, 0]), int(I["lists"][0, 1, 2])):
        idx = (e, 5)
        h = 1e-6
        Wp = dict(W); Wp["emb"] = W["emb"].copy(); Wp["emb"][idx] += h
        Wm = dict(W); Wm["emb"] = W["emb"].copy(); Wm["emb"][idx] -= h
        fd = (_loss_of(c, Wp, I, a, "ce") - _loss_of(c, Wm, I, a, "ce")) / (2 * h)
        assert abs(fd - g["emb"][idx]) <= 1e-6 * max(1e-3, abs(fd))


def test_losses_reduce_to_closed_forms():
    K, L = 6, 4
    s0 = torch.zeros(K)
    r = np.array([0, 1, 4, 2, 4, 3])
    # equal scores: CE = log K whatever the label; BCE = log 2 whatever the target
    assert float(train.request_loss("ce", s0, r, 2, L)) == pytest.approx(math.log(K), rel=1e-15)
    assert float(train.request_loss("bce", s0, r, 2, L)) == pytest.approx(math.log(2.0), rel=1e-15)
    # scores equal to the targets: MSE = 0
    assert float(train.request_loss("mse", torch.tensor(r, dtype=torch.float64), r, 2, L)) == 0.0
    # gradients: CE -> softmax(s) - e_y; BCE -> (sigma(s) - r/L) / K; MSE -> 2 (s - r) / K
    s = torch.tensor([0.3, -1.2, 2.0, 0.5, -0.4, 1.1], requires_grad=True)
    train.request_loss("ce", s, r, 2, L).backward()
    p = np.exp(s.detach().numpy()); p /= p.sum(); p[2] -= 1.0
    assert np.allclose(s.grad.numpy(), p, rtol=0, atol=1e-15)
    s.grad = None
    train.request_loss("bce", s, r, 2, L).backward()
    want = (1 / (1 + np.exp(-s.detach().numpy())) - r / L) / K
    assert np.allclose(s.grad.numpy(), want, rtol=0, atol=1e-15)
    s.grad = None
    train.request_loss("mse", s, r, 2, L).backward()
    assert np.allclose(s.grad.numpy(), 2 * (s.detach().numpy() - r) / K, rtol=0, atol=1e-15)


def test_labels_min_argmax_of_relevant_counts():
    lists = np.array([[[0, 1], [2, 3], [1, 2], [4, 0]]])
    relevant = np.array([[1, 0, 1, 1, 0]])
    r, y = train.sequence_labels(lists, relevant)
    assert r.tolist() == [[1, 2, 1, 1]]
    assert y.tolist() == [1]
    relevant = np.array([[0, 1, 1, 0, 0]])             # r = [1, 1, 2, 0]: unique max at k = 2
    assert train.sequence_labels(lists, relevant)[1].tolist() == [2]
    relevant = np.zeros((1, 5), dtype=np.int32)        # all ties: the smallest index
    assert train.sequence_labels(lists, relevant)[1].tolist() == [0]


def test_relevance_generator_is_seeded_and_binary():
    c = gen.config(1, B=3)
    a, b = gen.make_relevance(c), gen.make_relevance(c)
    assert a.shape == (3, c.M) and np.array_equal(a, b) and set(np.unique(a)) <= {0, 1}


def test_entries_outside_the_pool():
    """An entry outside [0, M): the same scores whatever its value (it is out of the distinct set and
    its row is a zero row), no feedback in the labels, and gradients that still equal finite
    differences (the position of that row gets nothing)."""
    c, W, I = _tiny(0, K=4, L=3, T=6, M=9)
    W = {k: np.asarray(v, np.float64) for k, v in W.items()}
    a = gen.make_relevance(c)
    a[0, :] = 1
    runs = []
    for bad in (c.M, c.M + 4, -1, -9):
        lists = I["lists"].copy()
        lists[0, 2, 1] = bad
        J = dict(I, lists=lists)
        r, _ = train.sequence_labels(lists, a)
        assert r[0, 2] == 2                             # every element relevant but the outside one
        P = {k: torch.tensor(v) for k, v in W.items()}
        runs.append((train.request_scores(c, P, J, 0).numpy(), J))
    for s_, _ in runs[1:]:
        assert np.array_equal(s_, runs[0][0])
    J = runs[0][1]
    _, g, _ = train.train_grads(c, W, J, a, "mse")
    for name, idx in (("pos", (2, 3)), ("pos", (1, 0)), ("item.0.w1", (3, 7)), ("cls", (5,))):
        h = 1e-6
        Wp = dict(W); Wp[name] = W[name].copy(); Wp[name][idx] += h
        Wm = dict(W); Wm[name] = W[name].copy(); Wm[name][idx] -= h
        fd = (_loss_of(c, Wp, J, a, "mse") - _loss_of(c, Wm, J, a, "mse")) / (2 * h)
        assert abs(fd - g[name][idx]) <= 1e-6 * max(1e-3, abs(fd)), (name, idx, fd, g[name][idx])
