"""Plain float64 CPU oracle of the FlashEvaluator joint-evaluation forward pass.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module: only the tests, the smoke check and the benchmark's CPU
baseline leg use it.  It shares no code with the HIP library; the seeded
input generator `gen` is the only module both sides read.

What is computed (paper, Sections 3 and 4):

  instance z = (x, C(x), L_1..L_K)                        (Section 3, problem statement)
  U(z)  = distinct elements of L_1..L_K                    (Section 4.1)
  H     = Enc(x, U(z)):  item-set self-attention, then cross-attention with
          the items as queries and the encoded context as keys/values (Section 4.2)
  c_k   = SeqEnc([CLS; H[L_k] + positions])                (Section 4.3)
  C'    = SelfAttn(c_1..c_K)                               (Section 4.4)
  s_k   = head(C'_k),   y = argmax_k s_k                   (Section 4.4; eq. (1))

The paper leaves the layer internals open; this oracle fixes them as follows
(the GPU path takes the same readings):
  * every attention module is standard multi-head attention with biases on
    the q/k/v/o projections and scale 1/sqrt(d_head);
  * blocks are pre-LayerNorm with residual connections, LayerNorm eps 1e-5
    with the biased variance, FFN = ReLU(x W1 + b1) W2 + b2;
  * the Query Context Module is n encoder blocks plus a final LayerNorm, no
    positional encoding; the key/value projections used by item layer l are
    applied to that encoded context once per request (the context-side
    key/value reuse of Section 4.2);
  * the item encoder is n blocks of [set self-attention, cross-attention to
    the context, FFN] plus a final LayerNorm;
  * SeqEnc and the cross-sequence module are n encoder blocks plus a final
    LayerNorm each, no mask; c_k is the final-normalised [CLS] row;
  * positions are added after the gather (Section 4.3), [CLS] sits at
    position 0; the head is a linear map to one scalar with bias;
  * selection takes the smallest index among the maximal scores (the
    min-argmax tie rule of the label construction, Appendix B.1); NaN scores
    never win and an all-NaN vector selects -1.

Linear-attention variant (cfg.attention == "linear"; the deployment setting
of Appendix B.3, which serves both evaluators with the kernelized attention
of the cited linear-attention work): the context self-attention, the items'
cross-attention to the context and the cross-sequence attention use
phi(q) . phi(k) weights with phi = elu + 1, no scale, normalised by their
sum; the item-set self-attention and SeqEnc keep softmax.

Two evaluation orders are provided:
  * `evaluate_naive` -- the oracle proper.  It follows the cost structure of
    the candidate-factorised evaluator (Section 4 and Appendix A.3): the
    context is encoded again for every candidate list, and the item-set
    encoding is recomputed for every item occurrence.  QKV-Cache is exact
    reuse (Section 4.2), so this must equal the joint pass.
  * `evaluate_cached` -- the same network with the context and item-set
    encodings computed once per request, which is the joint pass's order.
    Tests pin it to `evaluate_naive`; it is used where the naive order is too
    slow.

Conventions: row vectors times matrices; parameters are the dict produced by
`gen.make_weights` (float32 arrays whose values are upcast to float64 here).
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

LN_EPS = 1e-5

Params = Dict[str, np.ndarray]


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


# ---------------------------------------------------------------------------------------------
# Primitives
# ---------------------------------------------------------------------------------------------

def layer_norm(x: np.ndarray, g: np.ndarray, b: np.ndarray) -> np.ndarray:
    """LayerNorm over the last axis: g * (x - mean) / sqrt(var + eps) + b, biased variance."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return _f64(g) * (x - mu) / np.sqrt(var + LN_EPS) + _f64(b)


def softmax_rows(z: np.ndarray) -> np.ndarray:
    """exp(z - max z) / sum exp(z - max z) along the last axis."""
    z = z - z.max(axis=-1, keepdims=True)
    e = np.exp(z)
    return e / e.sum(axis=-1, keepdims=True)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, n_heads: int) -> np.ndarray:
    """Multi-head scaled dot-product attention on already projected q [nq,d], k, v [nk,d].

    Head h uses columns h*dh..(h+1)*dh-1; the heads' outputs are concatenated
    back in the same column order.  No mask: callers pass exactly the valid keys.
    """
    d = q.shape[-1]
    dh = d // n_heads
    out = np.empty((q.shape[0], d), dtype=np.float64)
    for h in range(n_heads):
        cols = slice(h * dh, (h + 1) * dh)
        a = softmax_rows(q[:, cols] @ k[:, cols].T / np.sqrt(dh))
        out[:, cols] = a @ v[:, cols]
    return out


def elu_plus_one(x: np.ndarray) -> np.ndarray:
    """Feature map of kernelized attention: phi(x) = elu(x) + 1, i.e. x + 1 for x > 0 and
    exp(x) otherwise (the map of the linear attention the paper's deployment uses, App. B.3)."""
    x = np.asarray(x, dtype=np.float64)
    return np.where(x > 0, x + 1.0, np.exp(np.minimum(x, 0.0)))


def linear_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, n_heads: int) -> np.ndarray:
    """Multi-head linear attention on already projected q [nq,d], k, v [nk,d], in its defining
    form: per head, the weight of key j for query i is phi(q_i) . phi(k_j), and the output is the
    weighted sum of the values divided by the sum of the weights.  No scale and no mask (callers
    pass exactly the valid keys)."""
    d = q.shape[-1]
    dh = d // n_heads
    out = np.empty((q.shape[0], d), dtype=np.float64)
    for h in range(n_heads):
        cols = slice(h * dh, (h + 1) * dh)
        w = elu_plus_one(q[:, cols]) @ elu_plus_one(k[:, cols]).T
        out[:, cols] = (w @ v[:, cols]) / w.sum(axis=1, keepdims=True)
    return out


def linear_kv_state(k: np.ndarray, v: np.ndarray, n_heads: int) -> np.ndarray:
    """Key/value cache of a linear-attention module: per head h, the sums over all keys t of
    phi(k_t) v_t^T (dh x dh) and of phi(k_t) (dh).  Returned as [n_heads][dh + 1][dh]: rows
    0..dh-1 hold the first sum (row i = feature i of phi(k)), row dh the second.  A query q then
    attends as (phi(q)^T S) / (phi(q) . z), which equals `linear_attention` by associativity."""
    d = k.shape[-1]
    dh = d // n_heads
    st = np.zeros((n_heads, dh + 1, dh), dtype=np.float64)
    for h in range(n_heads):
        cols = slice(h * dh, (h + 1) * dh)
        fk = elu_plus_one(k[:, cols])
        for t in range(k.shape[0]):
            st[h, :dh] += np.outer(fk[t], v[t, cols])
            st[h, dh] += fk[t]
    return st


def attend(q: np.ndarray, k: np.ndarray, v: np.ndarray, n_heads: int, kind: str = "softmax") -> np.ndarray:
    """Scaled dot-product attention (kind "softmax") or linear attention (kind "linear")."""
    if kind == "linear":
        return linear_attention(q, k, v, n_heads)
    if kind != "softmax":
        raise ValueError(f"unknown attention kind {kind!r}")
    return attention(q, k, v, n_heads)


def module_attention(cfg, module: str) -> str:
    """Attention kind of a module.  With cfg.attention == "linear", the attentions over sets
    whose size grows with the workload -- the context self-attention ("ctx"), the items'
    cross-attention to the context ("item_cross") and the cross-sequence attention over the K
    lists ("cross") -- are linear; the item-set self-attention ("item_self") and SeqEnc ("seq")
    stay softmax."""
    if getattr(cfg, "attention", "softmax") == "linear" and module in ("ctx", "item_cross", "cross"):
        return "linear"
    return "softmax"


def self_attention_block(x: np.ndarray, W: Params, p: str, n_heads: int, kind: str = "softmax") -> np.ndarray:
    """MHA(x, x) with the packed q|k|v projection `{p}.wqkv` and output projection `{p}.wo`."""
    d = x.shape[-1]
    qkv = x @ _f64(W[f"{p}.wqkv"]) + _f64(W[f"{p}.bqkv"])
    o = attend(qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:], n_heads, kind)
    return o @ _f64(W[f"{p}.wo"]) + _f64(W[f"{p}.bo"])


def ffn(x: np.ndarray, W: Params, p: str) -> np.ndarray:
    h = np.maximum(x @ _f64(W[f"{p}.w1"]) + _f64(W[f"{p}.b1"]), 0.0)
    return h @ _f64(W[f"{p}.w2"]) + _f64(W[f"{p}.b2"])


def encoder_block(x: np.ndarray, W: Params, p: str, n_heads: int, kind: str = "softmax") -> np.ndarray:
    """Pre-LN encoder block: x + MHA(LN1 x); then + FFN(LN2 x)."""
    x = x + self_attention_block(layer_norm(x, W[f"{p}.ln1.g"], W[f"{p}.ln1.b"]), W, p, n_heads, kind)
    x = x + ffn(layer_norm(x, W[f"{p}.ln2.g"], W[f"{p}.ln2.b"]), W, p)
    return x


def encoder_stack(x: np.ndarray, W: Params, module: str, n_layers: int, n_heads: int,
                  kind: str = "softmax") -> np.ndarray:
    """n pre-LN encoder blocks followed by the module's final LayerNorm."""
    for l in range(n_layers):
        x = encoder_block(x, W, f"{module}.{l}", n_heads, kind)
    return layer_norm(x, W[f"{module}.lnf.g"], W[f"{module}.lnf.b"])


# ---------------------------------------------------------------------------------------------
# Stages (one request)
# ---------------------------------------------------------------------------------------------

def context_rows(cfg, W: Params, inp: Dict, b: int) -> np.ndarray:
    """Context x of request b as rows; token-id contexts are embedded through E."""
    if cfg.vocab:
        return _f64(W["emb"])[inp["ctx_ids"][b]]
    return _f64(inp["x"][b])


def encode_context(cfg, W: Params, X: np.ndarray) -> Tuple[np.ndarray, List[Tuple[np.ndarray, np.ndarray]]]:
    """Query Context Module (Section 4.2) and the per-item-layer key/value cache.

    Returns the encoded context Q (T x d) and, for every item layer l,
    (K_l, V_l) = (Q Wk_l + bk_l, Q Wv_l + bv_l).
    """
    Q = encoder_stack(X, W, "ctx", cfg.n_layers, cfg.n_heads, module_attention(cfg, "ctx"))
    kv = []
    for l in range(cfg.n_layers):
        p = f"ctx.kv.{l}"
        kv.append((Q @ _f64(W[f"{p}.wk"]) + _f64(W[f"{p}.bk"]),
                   Q @ _f64(W[f"{p}.wv"]) + _f64(W[f"{p}.bv"])))
    return Q, kv


def distinct_items(lists_b: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """U(z) in ascending element id, and for every occurrence its rank in U(z) (Section 4.1)."""
    flat = [int(v) for v in np.asarray(lists_b).reshape(-1)]
    uniq = sorted(set(flat))
    rank = {v: r for r, v in enumerate(uniq)}
    slot = np.array([rank[v] for v in flat], dtype=np.int32).reshape(np.asarray(lists_b).shape)
    return np.array(uniq, dtype=np.int32), slot


def item_rows(cfg, W: Params, inp: Dict, b: int, uniq: np.ndarray) -> np.ndarray:
    """Element embeddings h_i for i in U(z): pool rows, or rows of E for token ids."""
    if cfg.vocab:
        return _f64(W["emb"])[uniq]
    return _f64(inp["pool"][b])[uniq]


def encode_items(cfg, W: Params, G: np.ndarray, kv: List[Tuple[np.ndarray, np.ndarray]]) -> np.ndarray:
    """Item-set encoder (Section 4.2): per layer set self-attention, cross-attention with the
    items as queries against the context cache, and FFN; then the final LayerNorm gives H."""
    for l in range(cfg.n_layers):
        p = f"item.{l}"
        G = G + self_attention_block(layer_norm(G, W[f"{p}.ln1.g"], W[f"{p}.ln1.b"]), W, p, cfg.n_heads,
                                     module_attention(cfg, "item_self"))
        q = layer_norm(G, W[f"{p}.ln2.g"], W[f"{p}.ln2.b"]) @ _f64(W[f"{p}.wq"]) + _f64(W[f"{p}.bq"])
        o = attend(q, kv[l][0], kv[l][1], cfg.n_heads, module_attention(cfg, "item_cross"))
        G = G + o @ _f64(W[f"{p}.wo2"]) + _f64(W[f"{p}.bo2"])
        h = layer_norm(G, W[f"{p}.ln3.g"], W[f"{p}.ln3.b"])
        G = G + np.maximum(h @ _f64(W[f"{p}.w1"]) + _f64(W[f"{p}.b1"]), 0.0) @ _f64(W[f"{p}.w2"]) \
            + _f64(W[f"{p}.b2"])
    return layer_norm(G, W["item.lnf.g"], W["item.lnf.b"])


def assemble_one(W: Params, rows: np.ndarray) -> np.ndarray:
    """[CLS; rows] with position p added to row p (positions after indexing, Section 4.3)."""
    L = rows.shape[0]
    pos = _f64(W["pos"])
    seq = np.empty((L + 1, rows.shape[1]), dtype=np.float64)
    seq[0] = _f64(W["cls"]) + pos[0]
    seq[1:] = rows + pos[1:L + 1]
    return seq


def encode_sequence(cfg, W: Params, seq: np.ndarray) -> np.ndarray:
    """SeqEnc over one assembled list; c_k is the final-normalised [CLS] row (Section 4.3)."""
    return encoder_stack(seq, W, "seq", cfg.n_layers, cfg.n_heads, module_attention(cfg, "seq"))[0]


def cross_sequence(cfg, W: Params, c: np.ndarray) -> np.ndarray:
    """Self-attention over the set {c_1..c_K} with no positions (Section 4.4)."""
    return encoder_stack(c, W, "cross", cfg.n_layers, cfg.n_heads, module_attention(cfg, "cross"))


def score(W: Params, Cp: np.ndarray) -> np.ndarray:
    """Shared linear prediction head s_k = C'_k . w + b (Section 4.4)."""
    return Cp @ _f64(W["head.w"]) + _f64(W["head.b"])[0]


def score_objectives(Cp: np.ndarray, head_w: np.ndarray, head_b: np.ndarray,
                     fuse_w: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Multi-objective head (Section 4.4): task heads s^t_k = C'_k . w_t + b_t on the shared C'_k,
    fused into s_k = sum_t alpha_t s^t_k.  The paper leaves the fusion module open; this reading
    is a weighted sum with given weights.  Returns (per-task scores [K][n_obj], fused [K])."""
    obj = Cp @ _f64(head_w).T + _f64(head_b)
    return obj, obj @ _f64(fuse_w)


def select(s: np.ndarray) -> int:
    """argmax_k s_k (eq. (1)); smallest index among ties; NaN never selected; all NaN -> -1."""
    best, best_v = -1, None
    for k, v in enumerate(np.asarray(s, dtype=np.float64)):
        if np.isnan(v):
            continue
        if best_v is None or v > best_v:
            best, best_v = k, v
    return best


# ---------------------------------------------------------------------------------------------
# Whole pass
# ---------------------------------------------------------------------------------------------

def _requests(cfg, requests: Optional[Sequence[int]]) -> List[int]:
    return list(range(cfg.B)) if requests is None else [int(b) for b in requests]


def evaluate_naive(cfg, W: Params, inp: Dict, requests: Optional[Sequence[int]] = None,
                   lists_limit: Optional[int] = None, cross_seq: bool = True) -> Dict[int, Dict[str, np.ndarray]]:
    """The oracle: candidate-factorised recomputation of the joint network.

    For every list k the context is encoded again; for every occurrence
    (k, j) the whole item-set encoding is recomputed and the row of element
    lists[k][j] is taken from it.  Only the cross-sequence module, which acts
    on all K lists at once, runs once per request.  `lists_limit` stops after
    that many lists (used to time a bounded sample; scores are then absent).
    `cross_seq=False` is the variant without cross-sequence interaction
    (the "- CrossSeq" ablation of Appendix B.4): C' = c, each list scored on
    its own representation.
    """
    out = {}
    for b in _requests(cfg, requests):
        lists_b = np.asarray(inp["lists"][b])
        K, L = lists_b.shape
        n_lists = K if lists_limit is None else min(K, lists_limit)
        c = np.empty((n_lists, cfg.d), dtype=np.float64)
        for k in range(n_lists):
            _, kv = encode_context(cfg, W, context_rows(cfg, W, inp, b))
            rows = np.empty((L, cfg.d), dtype=np.float64)
            for j in range(L):
                uniq, _ = distinct_items(lists_b)
                H = encode_items(cfg, W, item_rows(cfg, W, inp, b, uniq), kv)
                rows[j] = H[int(np.searchsorted(uniq, lists_b[k, j]))]
            c[k] = encode_sequence(cfg, W, assemble_one(W, rows))
        res = {"c": c}
        if n_lists == K:
            Cp = cross_sequence(cfg, W, c) if cross_seq else c
            s = score(W, Cp)
            res.update(Cp=Cp, scores=s, best=select(s))
        out[b] = res
    return out


def evaluate_cached(cfg, W: Params, inp: Dict, requests: Optional[Sequence[int]] = None,
                    stages: bool = False, cross_seq: bool = True) -> Dict[int, Dict[str, np.ndarray]]:
    """The same network in the joint pass's order: context and item set encoded once.

    With `stages=True` every intermediate is returned too: kv (list of
    (K_l, V_l)), uniq, slot, H (U x d), seq (K x (L+1) x d).  `cross_seq`
    as in `evaluate_naive`.
    """
    out = {}
    for b in _requests(cfg, requests):
        lists_b = np.asarray(inp["lists"][b])
        K, L = lists_b.shape
        _, kv = encode_context(cfg, W, context_rows(cfg, W, inp, b))
        uniq, slot = distinct_items(lists_b)
        H = encode_items(cfg, W, item_rows(cfg, W, inp, b, uniq), kv)
        seq = np.stack([assemble_one(W, H[slot[k]]) for k in range(K)])
        c = np.stack([encode_sequence(cfg, W, seq[k]) for k in range(K)])
        Cp = cross_sequence(cfg, W, c) if cross_seq else c
        s = score(W, Cp)
        res = {"c": c, "Cp": Cp, "scores": s, "best": select(s)}
        if stages:
            res.update(kv=kv, uniq=uniq, slot=slot, H=H, seq=seq)
        out[b] = res
    return out
