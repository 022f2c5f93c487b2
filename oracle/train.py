"""Plain float64 reference of the training step (Section 4.5, Appendix B.1).

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or execute this module:
only the tests and the benchmark use it.  It shares no code with the HIP library.

It writes the joint pass's forward out again in torch (float64, the same readings as
`oracle.evaluator`, which the tests pin it to) so that reverse-mode differentiation gives the
gradient of the batch loss with respect to every parameter.  The losses are those of Section 4.5:

  MSE  = (1/K) sum_k (s_k - s*_k)^2
  BCE  = -(1/K) sum_k [ s*_k log sigma(s_k) + (1 - s*_k) log(1 - sigma(s_k)) ]
  CE   = -log( exp(s_y) / sum_k exp(s_k) )

per request, averaged over the B requests of the batch.  Labels follow Appendix B.1: with a_{k,j}
the binary feedback of the j-th element of list k, r_k = sum_j a_{k,j} and y = the smallest k that
attains max r_k.  The scalar target of the MSE reading is r_k, the probabilistic target of the BCE
reading r_k / L.
"""
from __future__ import annotations

from typing import Dict, Optional, Tuple

import numpy as np
import torch

from .evaluator import LN_EPS, distinct_items

LOSSES = ("mse", "bce", "ce")


def sequence_labels(lists: np.ndarray, relevant: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """r[b][k] = sum_j relevant[b][lists[b][k][j]] and y[b] = min argmax_k r[b][k] (App. B.1).
    An entry outside the pool [0, M) has no feedback (it adds 0)."""
    lists = np.asarray(lists)
    B, K, L = lists.shape
    M = np.asarray(relevant).shape[1]
    r = np.zeros((B, K), dtype=np.int64)
    y = np.zeros(B, dtype=np.int64)
    for b in range(B):
        for k in range(K):
            r[b, k] = sum(int(relevant[b][int(e)]) for e in lists[b, k] if 0 <= int(e) < M)
        best = 0
        for k in range(1, K):
            if r[b, k] > r[b, best]:
                best = k
        y[b] = best
    return r, y


def _ln(x, g, b):
    mu = x.mean(-1, keepdim=True)
    var = ((x - mu) ** 2).mean(-1, keepdim=True)
    return g * (x - mu) / torch.sqrt(var + LN_EPS) + b


def _mha(q, k, v, H):
    d = q.shape[-1]
    dh = d // H
    outs = []
    for h in range(H):
        c = slice(h * dh, (h + 1) * dh)
        a = torch.softmax(q[:, c] @ k[:, c].T / np.sqrt(dh), dim=-1)
        outs.append(a @ v[:, c])
    return torch.cat(outs, dim=-1)


def _self_attn(x, P, p, H):
    d = x.shape[-1]
    qkv = x @ P[f"{p}.wqkv"] + P[f"{p}.bqkv"]
    return _mha(qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:], H) @ P[f"{p}.wo"] + P[f"{p}.bo"]


def _ffn(x, P, p):
    return torch.relu(x @ P[f"{p}.w1"] + P[f"{p}.b1"]) @ P[f"{p}.w2"] + P[f"{p}.b2"]


def _stack(x, P, module, n, H):
    for l in range(n):
        p = f"{module}.{l}"
        x = x + _self_attn(_ln(x, P[f"{p}.ln1.g"], P[f"{p}.ln1.b"]), P, p, H)
        x = x + _ffn(_ln(x, P[f"{p}.ln2.g"], P[f"{p}.ln2.b"]), P, p)
    return _ln(x, P[f"{module}.lnf.g"], P[f"{module}.lnf.b"])


def request_scores(cfg, P: Dict[str, torch.Tensor], inp: Dict, b: int) -> torch.Tensor:
    """s_1..s_K of request b: the joint pass (Sections 4.1-4.4) in the cached order.

    A list entry outside the pool [0, M) is left out of the distinct set and its sequence row is
    a zero row without a position (the reading the GPU step takes for such entries)."""
    if getattr(cfg, "attention", "softmax") != "softmax":
        raise NotImplementedError("the training reference covers softmax attention")
    n, H = cfg.n_layers, cfg.n_heads
    X = P["emb"][torch.as_tensor(inp["ctx_ids"][b], dtype=torch.long)] if cfg.vocab else \
        torch.as_tensor(np.asarray(inp["x"][b], np.float64))
    Q = _stack(X, P, "ctx", n, H)
    lists_b = np.asarray(inp["lists"][b])
    K, L = lists_b.shape
    valid = (lists_b >= 0) & (lists_b < cfg.M)
    uniq, _ = distinct_items(lists_b[valid])
    rank = {int(v): i for i, v in enumerate(uniq)}
    slot = np.array([[rank[int(e)] if ok else -1 for e, ok in zip(lists_b[k], valid[k])] for k in range(K)])
    idx = torch.as_tensor(uniq, dtype=torch.long)
    G = P["emb"][idx] if cfg.vocab else torch.as_tensor(np.asarray(inp["pool"][b], np.float64))[idx]
    for l in range(n):
        p = f"item.{l}"
        Kl = Q @ P[f"ctx.kv.{l}.wk"] + P[f"ctx.kv.{l}.bk"]
        Vl = Q @ P[f"ctx.kv.{l}.wv"] + P[f"ctx.kv.{l}.bv"]
        G = G + _self_attn(_ln(G, P[f"{p}.ln1.g"], P[f"{p}.ln1.b"]), P, p, H)
        q = _ln(G, P[f"{p}.ln2.g"], P[f"{p}.ln2.b"]) @ P[f"{p}.wq"] + P[f"{p}.bq"]
        G = G + _mha(q, Kl, Vl, H) @ P[f"{p}.wo2"] + P[f"{p}.bo2"]
        G = G + _ffn(_ln(G, P[f"{p}.ln3.g"], P[f"{p}.ln3.b"]), P, p)
    Hm = _ln(G, P["item.lnf.g"], P["item.lnf.b"])
    pos = P["pos"]
    c = []
    for k in range(K):
        ok = torch.as_tensor(slot[k] >= 0)[:, None]
        rows = Hm[torch.as_tensor(np.maximum(slot[k], 0), dtype=torch.long)] + pos[1:L + 1]
        rows = torch.where(ok, rows, torch.zeros_like(rows))
        seq = torch.cat([(P["cls"] + pos[0])[None, :], rows], dim=0)
        c.append(_stack(seq, P, "seq", n, H)[0])
    Cp = _stack(torch.stack(c), P, "cross", n, H)
    return Cp @ P["head.w"] + P["head.b"][0]


def request_loss(kind: str, s: torch.Tensor, r: np.ndarray, y: int, L: int) -> torch.Tensor:
    """Section 4.5 losses of one request from its scores s [K]."""
    if kind == "mse":
        t = torch.as_tensor(np.asarray(r, np.float64))
        return ((s - t) ** 2).mean()
    if kind == "bce":
        t = torch.as_tensor(np.asarray(r, np.float64) / L)
        # log sigma(s) = -softplus(-s), log(1 - sigma(s)) = -softplus(s)
        return (t * torch.nn.functional.softplus(-s) + (1 - t) * torch.nn.functional.softplus(s)).mean()
    if kind == "ce":
        return torch.logsumexp(s, dim=0) - s[int(y)]
    raise ValueError(kind)


def train_grads(cfg, W: Dict[str, np.ndarray], inp: Dict, relevant: np.ndarray, kind: str,
                requests: Optional[list] = None) -> Tuple[float, Dict[str, np.ndarray], np.ndarray]:
    """Batch loss (mean of the requests' losses), its gradient for every parameter, and the scores.

    `requests` restricts the batch to those requests (the loss is then their mean)."""
    P = {k: torch.tensor(np.asarray(v, np.float64), requires_grad=True) for k, v in W.items()}
    r, y = sequence_labels(inp["lists"], relevant)
    reqs = list(range(cfg.B)) if requests is None else list(requests)
    total = 0.0
    scores = []
    for b in reqs:
        s = request_scores(cfg, P, inp, b)
        scores.append(s.detach().numpy())
        total = total + request_loss(kind, s, r[b], y[b], cfg.L)
    loss = total / len(reqs)
    loss.backward()
    return float(loss.detach()), {k: P[k].grad.numpy().copy() for k in P}, np.stack(scores)
