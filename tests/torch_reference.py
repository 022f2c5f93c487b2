"""The joint-evaluation network assembled from torch.nn library layers (CPU, float64).

Used only to pin the numpy oracle: torch's TransformerEncoderLayer /
TransformerDecoderLayer (pre-LN, ReLU FFN, biased MHA, eps 1e-5) are an
implementation of the block definitions that was not written here.  The
oracle's parameters are loaded into them; torch stores linear weights as
[out, in], i.e. the transpose of the oracle's [in, out] matrices.
"""
from __future__ import annotations

import numpy as np
import torch
from torch import nn


def _t(a) -> torch.Tensor:
    return torch.as_tensor(np.asarray(a, dtype=np.float64))


def _ln(W, name: str, d: int) -> nn.LayerNorm:
    m = nn.LayerNorm(d, eps=1e-5, dtype=torch.float64)
    with torch.no_grad():
        m.weight.copy_(_t(W[f"{name}.g"]))
        m.bias.copy_(_t(W[f"{name}.b"]))
    return m


def encoder_layer(W, p: str, d: int, n_heads: int, F: int) -> nn.TransformerEncoderLayer:
    m = nn.TransformerEncoderLayer(d, n_heads, F, dropout=0.0, activation="relu", layer_norm_eps=1e-5,
                                   batch_first=True, norm_first=True, dtype=torch.float64)
    with torch.no_grad():
        m.self_attn.in_proj_weight.copy_(_t(W[f"{p}.wqkv"]).T)
        m.self_attn.in_proj_bias.copy_(_t(W[f"{p}.bqkv"]))
        m.self_attn.out_proj.weight.copy_(_t(W[f"{p}.wo"]).T)
        m.self_attn.out_proj.bias.copy_(_t(W[f"{p}.bo"]))
        m.linear1.weight.copy_(_t(W[f"{p}.w1"]).T)
        m.linear1.bias.copy_(_t(W[f"{p}.b1"]))
        m.linear2.weight.copy_(_t(W[f"{p}.w2"]).T)
        m.linear2.bias.copy_(_t(W[f"{p}.b2"]))
        m.norm1.weight.copy_(_t(W[f"{p}.ln1.g"]))
        m.norm1.bias.copy_(_t(W[f"{p}.ln1.b"]))
        m.norm2.weight.copy_(_t(W[f"{p}.ln2.g"]))
        m.norm2.bias.copy_(_t(W[f"{p}.ln2.b"]))
    return m.eval()


def decoder_layer(W, l: int, d: int, n_heads: int, F: int) -> nn.TransformerDecoderLayer:
    """Item layer l: set self-attention, cross-attention to the encoded context, FFN.

    The cross-attention's key/value projections are the context-side
    ctx.kv.{l}.wk / wv, applied by torch to `memory` (the encoded context).
    """
    p = f"item.{l}"
    m = nn.TransformerDecoderLayer(d, n_heads, F, dropout=0.0, activation="relu", layer_norm_eps=1e-5,
                                   batch_first=True, norm_first=True, dtype=torch.float64)
    with torch.no_grad():
        m.self_attn.in_proj_weight.copy_(_t(W[f"{p}.wqkv"]).T)
        m.self_attn.in_proj_bias.copy_(_t(W[f"{p}.bqkv"]))
        m.self_attn.out_proj.weight.copy_(_t(W[f"{p}.wo"]).T)
        m.self_attn.out_proj.bias.copy_(_t(W[f"{p}.bo"]))
        wq, wk, wv = _t(W[f"{p}.wq"]), _t(W[f"ctx.kv.{l}.wk"]), _t(W[f"ctx.kv.{l}.wv"])
        m.multihead_attn.in_proj_weight.copy_(torch.cat([wq.T, wk.T, wv.T], 0))
        m.multihead_attn.in_proj_bias.copy_(torch.cat([_t(W[f"{p}.bq"]), _t(W[f"ctx.kv.{l}.bk"]),
                                                       _t(W[f"ctx.kv.{l}.bv"])]))
        m.multihead_attn.out_proj.weight.copy_(_t(W[f"{p}.wo2"]).T)
        m.multihead_attn.out_proj.bias.copy_(_t(W[f"{p}.bo2"]))
        m.linear1.weight.copy_(_t(W[f"{p}.w1"]).T)
        m.linear1.bias.copy_(_t(W[f"{p}.b1"]))
        m.linear2.weight.copy_(_t(W[f"{p}.w2"]).T)
        m.linear2.bias.copy_(_t(W[f"{p}.b2"]))
        for i in (1, 2, 3):
            getattr(m, f"norm{i}").weight.copy_(_t(W[f"{p}.ln{i}.g"]))
            getattr(m, f"norm{i}").bias.copy_(_t(W[f"{p}.ln{i}.b"]))
    return m.eval()


def _stack(W, module: str, x: torch.Tensor, cfg) -> torch.Tensor:
    for l in range(cfg.n_layers):
        x = encoder_layer(W, f"{module}.{l}", cfg.d, cfg.n_heads, cfg.ffn)(x)
    return _ln(W, f"{module}.lnf", cfg.d)(x)


@torch.no_grad()
def evaluate_torch(cfg, W, inp, b: int, cross_seq: bool = True):
    """Scores of request b.  Items are indexed with torch.unique (sorted) and gathered by inverse."""
    lists = torch.as_tensor(np.asarray(inp["lists"][b], dtype=np.int64))
    if cfg.vocab:
        X = _t(W["emb"])[torch.as_tensor(np.asarray(inp["ctx_ids"][b], dtype=np.int64))]
    else:
        X = _t(inp["x"][b])
    mem = _stack(W, "ctx", X[None], cfg)
    uniq, inv = torch.unique(lists, sorted=True, return_inverse=True)
    src = _t(W["emb"]) if cfg.vocab else _t(inp["pool"][b])
    G = src[uniq][None]
    for l in range(cfg.n_layers):
        G = decoder_layer(W, l, cfg.d, cfg.n_heads, cfg.ffn)(G, mem)
    H = _ln(W, "item.lnf", cfg.d)(G)[0]
    K, L = lists.shape
    pos = _t(W["pos"])
    seq = torch.cat([(_t(W["cls"]) + pos[0]).expand(K, 1, cfg.d), H[inv] + pos[1:L + 1]], dim=1)
    c = _stack(W, "seq", seq, cfg)[:, 0]
    Cp = _stack(W, "cross", c[None], cfg)[0] if cross_seq else c
    head = nn.Linear(cfg.d, 1, dtype=torch.float64)
    head.weight.copy_(_t(W["head.w"])[None])
    head.bias.copy_(_t(W["head.b"]))
    s = head(Cp)[:, 0]
    return {"H": H.numpy(), "c": c.numpy(), "Cp": Cp.numpy(), "scores": s.numpy()}
