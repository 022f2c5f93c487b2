"""Where the bf16 path's score error comes from: the network of the oracle with bf16 rounding
(round to nearest even) applied at the points where the GPU path stores a value in bf16, switched
on and off one point at a time.  An analysis script run by hand (not a test):

    python tests/bf16_error_model.py WORKLOAD [K] [REQUESTS]

prints, per variant, max|ds| / max|s_ref| of each request against the exact float64 oracle.
Rounding points (the bf16 values of the GPU path; accumulation itself is exact here):
  ln   LayerNorm outputs that feed a product          qkv  projected queries, keys, values
  p    softmax weights entering P V (normalised after the product, in full precision)
  o    attention outputs                              hid  FFN hidden activations
  res  residual stream between kernels (context and item modules of models with d <= 256)
  kv   the context key/value cache                    H    the item encodings
  seq  the assembled sequences
"""
from __future__ import annotations

import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import gen  # noqa: E402
from oracle import evaluator as O  # noqa: E402

POINTS = ("ln", "qkv", "p", "o", "hid", "res", "kv", "H", "seq")


def bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to bfloat16 (via float32, ties to even) and back."""
    f = np.asarray(x, np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


class Model:
    def __init__(self, cfg, W, points):
        self.c, self.W, self.on = cfg, W, set(points)
        self.wide = cfg.d >= 512

    def R(self, x, tag):
        return bf16(x) if tag in self.on else x

    def w(self, name):
        return np.asarray(self.W[name], np.float64)

    def ln(self, x, p):
        return self.R(O.layer_norm(x, self.W[f"{p}.g"], self.W[f"{p}.b"]), "ln")

    def attend(self, q, k, v):
        H = self.c.n_heads
        d = q.shape[-1]
        dh = d // H
        out = np.empty((q.shape[0], d))
        for h in range(H):
            c = slice(h * dh, (h + 1) * dh)
            z = q[:, c] @ k[:, c].T / np.sqrt(dh)
            e = np.exp(z - z.max(-1, keepdims=True))
            out[:, c] = (self.R(e, "p") @ v[:, c]) / e.sum(-1, keepdims=True)
        return self.R(out, "o")

    def self_attn(self, x, p):
        d = x.shape[-1]
        qkv = self.R(x @ self.w(f"{p}.wqkv") + self.w(f"{p}.bqkv"), "qkv")
        return self.attend(qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:]) @ self.w(f"{p}.wo") + self.w(f"{p}.bo")

    def ffn(self, x, p):
        h = self.R(np.maximum(x @ self.w(f"{p}.w1") + self.w(f"{p}.b1"), 0.0), "hid")
        return h @ self.w(f"{p}.w2") + self.w(f"{p}.b2")

    def stack(self, x, m, between):
        for l in range(self.c.n_layers):
            p = f"{m}.{l}"
            x = x + self.self_attn(self.ln(x, f"{p}.ln1"), p)
            x = x + self.ffn(self.ln(x, f"{p}.ln2"), p)
            if between:
                x = self.R(x, "res")
        return x

    def scores(self, I, b):
        c = self.c
        between = not self.wide            # fused kernels of d <= 256 models pass the residual in bf16
        X = self.w("emb")[I["ctx_ids"][b]] if c.vocab else np.asarray(I["x"][b], np.float64)
        Q = self.ln(self.stack(X, "ctx", between), "ctx.lnf")
        kv = [(self.R(Q @ self.w(f"ctx.kv.{l}.wk") + self.w(f"ctx.kv.{l}.bk"), "kv"),
               self.R(Q @ self.w(f"ctx.kv.{l}.wv") + self.w(f"ctx.kv.{l}.bv"), "kv")) for l in range(c.n_layers)]
        lists_b = np.asarray(I["lists"][b])
        uniq, slot = O.distinct_items(lists_b)
        G = self.w("emb")[uniq] if c.vocab else np.asarray(I["pool"][b], np.float64)[uniq]
        for l in range(c.n_layers):
            p = f"item.{l}"
            G = G + self.self_attn(self.ln(G, f"{p}.ln1"), p)
            if between:
                G = self.R(G, "res")
            q = self.R(self.ln(G, f"{p}.ln2") @ self.w(f"{p}.wq") + self.w(f"{p}.bq"), "qkv")
            G = G + self.attend(q, kv[l][0], kv[l][1]) @ self.w(f"{p}.wo2") + self.w(f"{p}.bo2")
            G = G + self.ffn(self.ln(G, f"{p}.ln3"), p)
            if between:
                G = self.R(G, "res")
        Hm = self.R(O.layer_norm(G, self.W["item.lnf.g"], self.W["item.lnf.b"]), "H")
        pos = self.w("pos")
        K, L = lists_b.shape
        cs = []
        for k in range(K):
            s = np.empty((L + 1, c.d))
            s[0] = self.w("cls") + pos[0]
            s[1:] = Hm[slot[k]] + pos[1:L + 1]
            s = self.stack(self.R(s, "seq"), "seq", False)
            cs.append(O.layer_norm(s, self.W["seq.lnf.g"], self.W["seq.lnf.b"])[0])
        Z = self.stack(np.stack(cs), "cross", False)
        return O.score(self.W, O.layer_norm(Z, self.W["cross.lnf.g"], self.W["cross.lnf.b"]))


def main() -> None:
    cid = int(sys.argv[1])
    K = int(sys.argv[2]) if len(sys.argv) > 2 and sys.argv[2] != "-" else None
    n = int(sys.argv[3]) if len(sys.argv) > 3 else 8
    c = gen.config(cid, K=K) if K else gen.config(cid)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    reqs = list(range(min(n, c.B)))
    ref = {b: r["scores"] for b, r in O.evaluate_cached(c, W, I, requests=reqs).items()}
    variants = [("all points", POINTS)] + [(f"all but {t}", [x for x in POINTS if x != t]) for t in POINTS]
    print(f"{c.label}: max|ds| / max|s_ref| over requests {reqs[0]}..{reqs[-1]}")
    for name, pts in variants:
        m = Model(c, W, pts)
        e = np.array([np.max(np.abs(m.scores(I, b) - ref[b])) / np.max(np.abs(ref[b])) for b in reqs])
        print(f"  {name:14s} max {e.max():.4f}  rms {np.sqrt(np.mean(e ** 2)):.4f}", flush=True)


if __name__ == "__main__":
    main()
