"""Parity at the edges of the supported envelope (include/flasheval.h): the longest context
(T = 8192), the most lists (K = 4096), the longest lists (L = 127, 128-row sequences) and the
largest pool (M = 131072), each on one request of the RecSys-base model, against the float64
oracle (cached order, pinned to the naive one on the CPU)."""
import numpy as np
import pytest

import gen
import oracle
from tests.gpu_harness import check_scores, normwise, rtol_for, run_pass

pytestmark = pytest.mark.gpu


def _check(c, W, I, out, kv=True):
    tol = rtol_for(c)
    ref = oracle.evaluate_cached(c, W, I, requests=[0], stages=True)[0]
    if kv:
        for l in range(c.n_layers):
            assert normwise(out["kv"][l, 0, 0], ref["kv"][l][0]) <= tol, ("K cache", l)
            assert normwise(out["kv"][l, 1, 0], ref["kv"][l][1]) <= tol, ("V cache", l)
    U = len(ref["uniq"])
    assert out["n_uniq"][0] == U
    assert np.array_equal(out["uniq"][0, :U], ref["uniq"])
    assert np.array_equal(out["slot"][0], ref["slot"])
    assert normwise(out["H"][0, :U], ref["H"]) <= tol, "H"
    assert normwise(out["seq"][0], ref["seq"]) <= tol, "seq"
    assert normwise(out["Cp"][0], ref["Cp"]) <= tol, "Cp"
    check_scores(c, out["scores"][0], out["best"][0], ref["scores"])
    assert np.all(out["status"] == 0)


def test_longest_context():
    c = gen.config(1, B=1, T=8192, K=4, L=5, M=20)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    _check(c, W, I, run_pass(c, W, I))


def test_most_lists():
    c = gen.config(1, B=1, T=16, K=4096, L=3, M=200)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    _check(c, W, I, run_pass(c, W, I))


def test_longest_lists():
    c = gen.config(1, B=1, T=16, K=3, L=127, M=300)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    _check(c, W, I, run_pass(c, W, I))


def test_largest_pool():
    c = gen.config(1, B=1, T=16, K=8, L=5, M=131072)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    _check(c, W, I, run_pass(c, W, I))


def test_longest_context_linear():
    """Linear attention over 8192 context rows: the state sums 8192 keys per head."""
    c = gen.config(1, B=1, T=8192, K=4, L=5, M=20, attention="linear")
    W, I = gen.make_weights(c), gen.make_inputs(c)
    out = run_pass(c, W, I)
    tol = rtol_for(c)
    ref = oracle.evaluate_cached(c, W, I, requests=[0], stages=True)[0]
    for l in range(c.n_layers):
        st = oracle.linear_kv_state(ref["kv"][l][0], ref["kv"][l][1], c.n_heads)
        assert normwise(out["kv"][l, 0], st) <= tol, ("linear state", l)
    assert normwise(out["Cp"][0], ref["Cp"]) <= tol, "Cp"
    check_scores(c, out["scores"][0], out["best"][0], ref["scores"])
