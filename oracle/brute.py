"""Scalar brute-force form of the joint-evaluation pass, for tiny inputs only.

TEST INFRASTRUCTURE ONLY (see oracle/evaluator.py).  This is a second,
independent spelling of the same network, written with plain Python lists,
explicit loops, math.exp and math.sqrt and no array library, so that a
mistake in the vectorised oracle (a transposed operand, a wrong head slice,
a dropped bias or residual) shows up as a disagreement.  It takes the same
parameter dict; numpy appears only to convert arrays to nested Python lists.
"""
from __future__ import annotations

import math
from typing import Dict, List

Vec = List[float]
Mat = List[List[float]]


def _tolist(a) -> list:
    return a.tolist() if hasattr(a, "tolist") else list(a)


def _vecmat(v: Vec, w: Mat, bias: Vec) -> Vec:
    """out[j] = sum_i v[i] * w[i][j] + bias[j]."""
    n_out = len(w[0])
    out = []
    for j in range(n_out):
        acc = 0.0
        for i in range(len(v)):
            acc += v[i] * w[i][j]
        out.append(acc + bias[j])
    return out


def _ln(v: Vec, g: Vec, b: Vec, eps: float = 1e-5) -> Vec:
    n = len(v)
    mean = sum(v) / n
    var = sum((t - mean) * (t - mean) for t in v) / n
    inv = 1.0 / math.sqrt(var + eps)
    return [g[i] * (v[i] - mean) * inv + b[i] for i in range(n)]


def _mha(qs: Mat, ks: Mat, vs: Mat, n_heads: int) -> Mat:
    """Per query row and head: softmax over keys of q.k/sqrt(dh), weighted sum of values."""
    d = len(qs[0])
    dh = d // n_heads
    scale = 1.0 / math.sqrt(dh)
    out = []
    for q in qs:
        row = [0.0] * d
        for h in range(n_heads):
            lo = h * dh
            logits = []
            for kk in ks:
                dot = 0.0
                for t in range(dh):
                    dot += q[lo + t] * kk[lo + t]
                logits.append(dot * scale)
            m = max(logits)
            ws = [math.exp(z - m) for z in logits]
            tot = sum(ws)
            for t in range(dh):
                acc = 0.0
                for r in range(len(vs)):
                    acc += ws[r] * vs[r][lo + t]
                row[lo + t] = acc / tot
        out.append(row)
    return out


def _phi(t: float) -> float:
    """elu(t) + 1."""
    return t + 1.0 if t > 0.0 else math.exp(t)


def _mha_linear(qs: Mat, ks: Mat, vs: Mat, n_heads: int) -> Mat:
    """Per query row and head: weight of key r = sum_t phi(q_t) phi(k_r,t); output = weighted sum
    of the values over the sum of the weights (kernelized attention, no scale)."""
    d = len(qs[0])
    dh = d // n_heads
    out = []
    for q in qs:
        row = [0.0] * d
        for h in range(n_heads):
            lo = h * dh
            ws = []
            for kk in ks:
                acc = 0.0
                for t in range(dh):
                    acc += _phi(q[lo + t]) * _phi(kk[lo + t])
                ws.append(acc)
            tot = sum(ws)
            for t in range(dh):
                acc = 0.0
                for r in range(len(vs)):
                    acc += ws[r] * vs[r][lo + t]
                row[lo + t] = acc / tot
        out.append(row)
    return out


class _P:
    def __init__(self, W: Dict):
        self.W = W

    def __getitem__(self, name):
        return _tolist(self.W[name])


def _self_attn(X: Mat, P: _P, p: str, n_heads: int, linear: bool = False) -> Mat:
    d = len(X[0])
    wqkv, bqkv = P[f"{p}.wqkv"], P[f"{p}.bqkv"]
    qkv = [_vecmat(x, wqkv, bqkv) for x in X]
    q = [r[:d] for r in qkv]
    k = [r[d:2 * d] for r in qkv]
    v = [r[2 * d:] for r in qkv]
    o = _mha_linear(q, k, v, n_heads) if linear else _mha(q, k, v, n_heads)
    return [_vecmat(r, P[f"{p}.wo"], P[f"{p}.bo"]) for r in o]


def _ffn(X: Mat, P: _P, p: str) -> Mat:
    out = []
    for x in X:
        h = [max(t, 0.0) for t in _vecmat(x, P[f"{p}.w1"], P[f"{p}.b1"])]
        out.append(_vecmat(h, P[f"{p}.w2"], P[f"{p}.b2"]))
    return out


def _add(A: Mat, B: Mat) -> Mat:
    return [[a + b for a, b in zip(ra, rb)] for ra, rb in zip(A, B)]


def _enc(X: Mat, P: _P, p: str, n_heads: int, linear: bool = False) -> Mat:
    Xn = [_ln(x, P[f"{p}.ln1.g"], P[f"{p}.ln1.b"]) for x in X]
    X = _add(X, _self_attn(Xn, P, p, n_heads, linear))
    Xn = [_ln(x, P[f"{p}.ln2.g"], P[f"{p}.ln2.b"]) for x in X]
    return _add(X, _ffn(Xn, P, p))


def _stack(X: Mat, P: _P, module: str, n_layers: int, n_heads: int, linear: bool = False) -> Mat:
    for l in range(n_layers):
        X = _enc(X, P, f"{module}.{l}", n_heads, linear)
    return [_ln(x, P[f"{module}.lnf.g"], P[f"{module}.lnf.b"]) for x in X]


def evaluate_brute(cfg, W: Dict, inp: Dict, b: int = 0) -> Dict:
    """Scores, selection and intermediates of request b, by explicit loops."""
    P = _P(W)
    nh, nl = cfg.n_heads, cfg.n_layers
    # linear-attention variant: context, item->context and cross-sequence attention are linear
    lin = getattr(cfg, "attention", "softmax") == "linear"
    if cfg.vocab:
        E = P["emb"]
        X = [list(E[t]) for t in _tolist(inp["ctx_ids"][b])]
    else:
        X = [list(r) for r in _tolist(inp["x"][b])]
    Q = _stack(X, P, "ctx", nl, nh, lin)
    kv = []
    for l in range(nl):
        p = f"ctx.kv.{l}"
        kv.append(([_vecmat(q, P[f"{p}.wk"], P[f"{p}.bk"]) for q in Q],
                   [_vecmat(q, P[f"{p}.wv"], P[f"{p}.bv"]) for q in Q]))
    lists_b = [[int(t) for t in row] for row in _tolist(inp["lists"][b])]
    seen = []
    for row in lists_b:
        for t in row:
            if t not in seen:
                seen.append(t)
    uniq = sorted(seen)
    src = P["emb"] if cfg.vocab else _tolist(inp["pool"][b])
    G = [list(src[i]) for i in uniq]
    for l in range(nl):
        p = f"item.{l}"
        Gn = [_ln(g, P[f"{p}.ln1.g"], P[f"{p}.ln1.b"]) for g in G]
        G = _add(G, _self_attn(Gn, P, p, nh))
        qs = [_vecmat(_ln(g, P[f"{p}.ln2.g"], P[f"{p}.ln2.b"]), P[f"{p}.wq"], P[f"{p}.bq"]) for g in G]
        o = _mha_linear(qs, kv[l][0], kv[l][1], nh) if lin else _mha(qs, kv[l][0], kv[l][1], nh)
        G = _add(G, [_vecmat(r, P[f"{p}.wo2"], P[f"{p}.bo2"]) for r in o])
        Gn = [_ln(g, P[f"{p}.ln3.g"], P[f"{p}.ln3.b"]) for g in G]
        G = _add(G, _ffn(Gn, P, p))
    H = [_ln(g, P["item.lnf.g"], P["item.lnf.b"]) for g in G]
    pos, cls = P["pos"], P["cls"]
    cs = []
    for row in lists_b:
        seq = [[cls[i] + pos[0][i] for i in range(len(cls))]]
        for j, t in enumerate(row):
            h = H[uniq.index(t)]
            seq.append([h[i] + pos[j + 1][i] for i in range(len(h))])
        cs.append(_stack(seq, P, "seq", nl, nh)[0])
    Cp = _stack(cs, P, "cross", nl, nh, lin)
    w, bias = P["head.w"], P["head.b"]
    scores = [sum(c[i] * w[i] for i in range(len(w))) + bias[0] for c in Cp]
    best = -1
    for k, s in enumerate(scores):
        if s == s and (best < 0 or s > scores[best]):
            best = k
    return {"uniq": uniq, "H": H, "c": cs, "Cp": Cp, "scores": scores, "best": best}
