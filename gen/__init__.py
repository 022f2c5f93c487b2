"""Seeded synthetic workloads for the FlashEvaluator joint-evaluation pass.

This module produces data only: configuration records, request inputs
(context x, candidate pool C(x), the K candidate lists L_1..L_K of the
problem statement in Section 3) and model parameters.  It contains none of
the evaluator's arithmetic, so both the CPU oracle and the GPU path can draw
their inputs from it without sharing any method code.

Everything is a numpy array.  Floating-point arrays are float32; for the
bf16 workloads every value is rounded to the nearest bfloat16 (ties to even)
before it is returned, so the same numbers are exactly representable in
both the bf16 device copy and the float64 oracle copy.

Workloads (numbered 0..4):

  0  tiny fp32 sanity        B=1,  T=16,   d=32,  H=1, n=1, M=20,   K=4,   L=5
  1  RecSys base             B=64, T=256,  d=128, H=4, n=2, M=200,  K=50,  L=10
  2  K sweep on workload 1   same as 1 with K in {10, 50, 200, 1000}
  3  long context            B=16, T=2048, d=256, H=8, n=2, M=500,  K=100, L=20
  4  text hypotheses         B=8,  T=1024, d=512, H=8, n=4, V=32000, K=16, L=64

Any workload can be taken with attention="linear" (the kernelized-attention
variant); the model parameters and inputs do not depend on that choice.

Sampling rules:
  * context and pool rows ~ N(0, 1) (workload 4: context rows are token ids
    uniform over the vocabulary, embedded by the model table E).
  * lists: workload 0 draws indices uniformly with repeats; workloads 1-3
    draw Zipf(s) ranks without repeats inside a list (successive
    renormalised draws), mapped to pool indices through a per-request
    random permutation; workload 4 draws one base hypothesis of L token ids
    per request and resamples each position with probability 0.2 for every
    one of the K hypotheses.
  * parameters ~ N(0, 0.02) for every matrix, bias, [CLS], learned position
    table, embedding table and score head; LayerNorm gains are 1 + N(0, 0.02)
    and LayerNorm offsets N(0, 0.02).  Workload 4 uses a fixed sinusoidal
    position table instead of a learned one.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field, replace
from typing import Dict, List, Optional, Tuple

import numpy as np

__all__ = [
    "Config", "config", "ALL_CONFIG_IDS", "K_SWEEP", "param_spec", "make_weights",
    "make_inputs", "round_bf16", "bf16_bits",
]

K_SWEEP = (10, 50, 200, 1000)


@dataclass(frozen=True)
class Config:
    """Shape and sampling record of one workload."""
    cid: int                 # workload number 0..4
    name: str
    B: int                   # requests per batch
    T: int                   # context rows per request
    d: int                   # model width
    n_heads: int
    n_layers: int            # layers in each of the four modules
    ffn: int                 # FFN hidden width
    M: int                   # pool size (workload 4: vocabulary size)
    K: int                   # candidate lists per request
    L: int                   # list length
    dtype: str               # "f32" or "bf16"
    list_kind: str           # "uniform", "zipf" or "text"
    zipf_s: float = 0.0
    vocab: int = 0           # >0: items and context are token ids into E[vocab][d]
    pos_kind: str = "learned"  # "learned" or "sinusoid"
    attention: str = "softmax"  # "softmax", or "linear": kernelized attention in the context,
                                # item->context and cross-sequence modules
    weight_seed: int = 0
    input_seed: int = 0
    list_seed: int = 0

    @property
    def dh(self) -> int:
        return self.d // self.n_heads

    @property
    def S(self) -> int:
        """Sequence length inside SeqEnc: [CLS] plus L items."""
        return self.L + 1

    @property
    def max_L(self) -> int:
        return self.L

    @property
    def U_cap(self) -> int:
        """Upper bound on distinct items per request."""
        return min(self.M, self.K * self.L)

    @property
    def label(self) -> str:
        return f"cfg{self.cid}" + (f"_K{self.K}" if self.cid == 2 else "") + \
            ("_linear" if self.attention == "linear" else "")


_BASE = {
    0: dict(name="tiny fp32 sanity", B=1, T=16, d=32, n_heads=1, n_layers=1, ffn=128, M=20, K=4, L=5,
            dtype="f32", list_kind="uniform"),
    1: dict(name="RecSys base", B=64, T=256, d=128, n_heads=4, n_layers=2, ffn=512, M=200, K=50, L=10,
            dtype="bf16", list_kind="zipf", zipf_s=1.1),
    3: dict(name="long context", B=16, T=2048, d=256, n_heads=8, n_layers=2, ffn=1024, M=500, K=100, L=20,
            dtype="bf16", list_kind="zipf", zipf_s=1.05),
    4: dict(name="text hypotheses", B=8, T=1024, d=512, n_heads=8, n_layers=4, ffn=2048, M=32000, K=16, L=64,
            dtype="bf16", list_kind="text", vocab=32000, pos_kind="sinusoid"),
}

ALL_CONFIG_IDS = (0, 1, 2, 3, 4)


def config(cid: int, K: Optional[int] = None, **overrides) -> Config:
    """Return workload `cid`.  Workload 2 takes K from K_SWEEP (default 50).

    Workload 2 reuses workload 1's model and its context/pool draws; only the
    lists (and their seed) depend on K.  `overrides` replace any field, which
    tests use to build reduced variants (e.g. B=2) that keep all other draws.
    """
    if cid == 2:
        k = 50 if K is None else int(K)
        if k not in K_SWEEP:
            raise ValueError(f"workload 2 takes K in {K_SWEEP}, got {k}")
        base = dict(_BASE[1], name=f"K sweep on RecSys base (K={k})", K=k)
        cfg = Config(cid=2, weight_seed=10_001, input_seed=20_001, list_seed=30_002 + k, **base)
    elif cid in _BASE:
        if K is not None:
            overrides = dict(overrides, K=int(K))
        cfg = Config(cid=cid, weight_seed=10_000 + cid, input_seed=20_000 + cid, list_seed=30_000 + cid,
                     **_BASE[cid])
    else:
        raise ValueError(f"unknown workload {cid}")
    if overrides:
        cfg = replace(cfg, **overrides)
    if cfg.d % cfg.n_heads:
        raise ValueError("d must be a multiple of n_heads")
    if cfg.attention not in ("softmax", "linear"):
        raise ValueError(f"attention must be 'softmax' or 'linear', got {cfg.attention!r}")
    return cfg


# --------------------------------------------------------------------------------------------
# bfloat16 rounding of generated values (input preparation, not evaluator arithmetic)
# --------------------------------------------------------------------------------------------

def bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16, ties to even; return the raw uint16 patterns."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    nan = (u & np.uint32(0x7FFFFFFF)) > np.uint32(0x7F800000)
    r = np.where(nan, (u >> np.uint32(16)) | np.uint32(0x40), r)
    return r.astype(np.uint16)


def round_bf16(a: np.ndarray) -> np.ndarray:
    """float32 array whose values are the bfloat16-rounded values of `a`."""
    return (bf16_bits(a).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _finish(cfg: Config, a: np.ndarray) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.float32)
    return round_bf16(a) if cfg.dtype == "bf16" else a


# --------------------------------------------------------------------------------------------
# Parameters
# --------------------------------------------------------------------------------------------

def _enc_block(prefix: str, d: int, F: int) -> List[Tuple[str, Tuple[int, ...], str]]:
    return [
        (f"{prefix}.ln1.g", (d,), "gain"), (f"{prefix}.ln1.b", (d,), "w"),
        (f"{prefix}.wqkv", (d, 3 * d), "w"), (f"{prefix}.bqkv", (3 * d,), "w"),
        (f"{prefix}.wo", (d, d), "w"), (f"{prefix}.bo", (d,), "w"),
        (f"{prefix}.ln2.g", (d,), "gain"), (f"{prefix}.ln2.b", (d,), "w"),
        (f"{prefix}.w1", (d, F), "w"), (f"{prefix}.b1", (F,), "w"),
        (f"{prefix}.w2", (F, d), "w"), (f"{prefix}.b2", (d,), "w"),
    ]


def param_spec(cfg: Config) -> List[Tuple[str, Tuple[int, ...], str]]:
    """Ordered (name, shape, init-kind) list of every model parameter.

    Matrices are stored in "input x output" orientation (a row vector times
    the matrix).  In wqkv the query, key and value projections are the three
    consecutive column blocks of width d; head h owns columns h*dh..(h+1)*dh-1
    inside each block.  The cross-attention key/value projections of item
    layer l ("ctx.kv.{l}.*") belong to the context side because they act on
    the encoded context, once per request.
    """
    d, F, n = cfg.d, cfg.ffn, cfg.n_layers
    spec: List[Tuple[str, Tuple[int, ...], str]] = []
    for l in range(n):
        spec += _enc_block(f"ctx.{l}", d, F)
    spec += [("ctx.lnf.g", (d,), "gain"), ("ctx.lnf.b", (d,), "w")]
    for l in range(n):
        spec += [(f"ctx.kv.{l}.wk", (d, d), "w"), (f"ctx.kv.{l}.bk", (d,), "w"),
                 (f"ctx.kv.{l}.wv", (d, d), "w"), (f"ctx.kv.{l}.bv", (d,), "w")]
    for l in range(n):
        p = f"item.{l}"
        spec += [
            (f"{p}.ln1.g", (d,), "gain"), (f"{p}.ln1.b", (d,), "w"),
            (f"{p}.wqkv", (d, 3 * d), "w"), (f"{p}.bqkv", (3 * d,), "w"),
            (f"{p}.wo", (d, d), "w"), (f"{p}.bo", (d,), "w"),
            (f"{p}.ln2.g", (d,), "gain"), (f"{p}.ln2.b", (d,), "w"),
            (f"{p}.wq", (d, d), "w"), (f"{p}.bq", (d,), "w"),
            (f"{p}.wo2", (d, d), "w"), (f"{p}.bo2", (d,), "w"),
            (f"{p}.ln3.g", (d,), "gain"), (f"{p}.ln3.b", (d,), "w"),
            (f"{p}.w1", (d, F), "w"), (f"{p}.b1", (F,), "w"),
            (f"{p}.w2", (F, d), "w"), (f"{p}.b2", (d,), "w"),
        ]
    spec += [("item.lnf.g", (d,), "gain"), ("item.lnf.b", (d,), "w")]
    for l in range(n):
        spec += _enc_block(f"seq.{l}", d, F)
    spec += [("seq.lnf.g", (d,), "gain"), ("seq.lnf.b", (d,), "w")]
    for l in range(n):
        spec += _enc_block(f"cross.{l}", d, F)
    spec += [("cross.lnf.g", (d,), "gain"), ("cross.lnf.b", (d,), "w")]
    spec += [("cls", (d,), "w"),
             ("pos", (cfg.max_L + 1, d), "sinusoid" if cfg.pos_kind == "sinusoid" else "w"),
             ("head.w", (d,), "w"), ("head.b", (1,), "w")]
    if cfg.vocab:
        spec += [("emb", (cfg.vocab, d), "w")]
    return spec


def _sinusoid_table(rows: int, d: int) -> np.ndarray:
    """Fixed position table: even column 2i holds sin(p / 10000^(2i/d)), odd column 2i+1 the cos."""
    p = np.arange(rows, dtype=np.float64)[:, None]
    i2 = np.arange(0, d, 2, dtype=np.float64)[None, :]
    ang = p / np.power(10000.0, i2 / d)
    t = np.zeros((rows, d), dtype=np.float64)
    t[:, 0::2] = np.sin(ang)
    t[:, 1::2] = np.cos(ang)
    return t


def make_weights(cfg: Config) -> Dict[str, np.ndarray]:
    """Draw every parameter in `param_spec` order from one seeded generator."""
    rng = np.random.default_rng(cfg.weight_seed)
    out: Dict[str, np.ndarray] = {}
    for name, shape, kind in param_spec(cfg):
        if kind == "gain":
            v = 1.0 + 0.02 * rng.standard_normal(shape, dtype=np.float32)
        elif kind == "sinusoid":
            v = _sinusoid_table(*shape)
        else:
            v = 0.02 * rng.standard_normal(shape, dtype=np.float32)
        out[name] = _finish(cfg, v)
    return out


# --------------------------------------------------------------------------------------------
# Inputs
# --------------------------------------------------------------------------------------------

def _zipf_lists(rng: np.random.Generator, B: int, M: int, K: int, L: int, s: float) -> np.ndarray:
    """Zipf(s) over pool ranks, no repeats inside a list, per-request rank->index permutation."""
    p = np.arange(1, M + 1, dtype=np.float64) ** (-s)
    p /= p.sum()
    out = np.empty((B, K, L), dtype=np.int32)
    for b in range(B):
        perm = rng.permutation(M)
        for k in range(K):
            out[b, k] = perm[rng.choice(M, L, replace=False, p=p)]
    return out


def _text_lists(rng: np.random.Generator, B: int, V: int, K: int, L: int, p_resample: float = 0.2) -> np.ndarray:
    out = np.empty((B, K, L), dtype=np.int32)
    for b in range(B):
        base = rng.integers(0, V, L)
        for k in range(K):
            h = base.copy()
            m = rng.random(L) < p_resample
            h[m] = rng.integers(0, V, int(m.sum()))
            out[b, k] = h
    return out


def make_inputs(cfg: Config) -> Dict[str, Optional[np.ndarray]]:
    """Return {"x": [B][T][d] or None, "ctx_ids": [B][T] or None, "pool": [B][M][d] or None,
    "lists": [B][K][L] int32}.  Workload 4 has token-id context and no pool."""
    rng = np.random.default_rng(cfg.input_seed)
    B, T, d, M, K, L = cfg.B, cfg.T, cfg.d, cfg.M, cfg.K, cfg.L
    if cfg.vocab:
        ctx_ids = rng.integers(0, cfg.vocab, (B, T)).astype(np.int32)
        x = None
        pool = None
    else:
        ctx_ids = None
        x = _finish(cfg, rng.standard_normal((B, T, d), dtype=np.float32))
        pool = _finish(cfg, rng.standard_normal((B, M, d), dtype=np.float32))
    lrng = np.random.default_rng(cfg.list_seed)
    if cfg.list_kind == "uniform":
        lists = lrng.integers(0, M, (B, K, L)).astype(np.int32)
    elif cfg.list_kind == "zipf":
        lists = _zipf_lists(lrng, B, M, K, L, cfg.zipf_s)
    elif cfg.list_kind == "text":
        lists = _text_lists(lrng, B, cfg.vocab, K, L)
    else:
        raise ValueError(cfg.list_kind)
    return {"x": x, "ctx_ids": ctx_ids, "pool": pool, "lists": lists}


def make_relevance(cfg: Config, p: float = 0.2, seed_offset: int = 40_000) -> np.ndarray:
    """Synthetic item-level feedback for training: a[b][m] in {0, 1}, Bernoulli(p) per request
    and element (int32 [B][M]; M = vocab for token-id items).  The labels built from it are the
    consumer's business."""
    rng = np.random.default_rng(seed_offset + cfg.cid + 97 * cfg.list_seed)
    return (rng.random((cfg.B, cfg.M)) < p).astype(np.int32)
