"""Helpers for GPU tests: upload a generated workload, run the five C-ABI calls, fetch results,
and compare them with the float64 oracle.

Tolerances (normwise per request and tensor, max|gpu - ref| <= rtol * max|ref|):
  * every float tensor (key/value cache, H, seq, C'): rtol 1e-4 for fp32 models and 2e-2 for
    bf16 models (bf16 operands, fp32 accumulation);
  * scores: rtol 1e-4 for fp32 models; bf16 models take SCORE_RTOL["bf16"] = 3e-2.  A score is
    a d-term dot product whose terms largely cancel (|s| is several times smaller than
    sum_i |C'_i w_i|), so the bf16 roundings of the whole network reach it relatively
    amplified: over every request of the five workloads the measured worst case of
    max|ds| / max|s_ref| is 2.27e-2 (text-hypothesis and K = 10 workloads), the typical case
    0.9e-2.  3e-2 is that measured bound with a 1.3x margin;
  * selection: the list the GPU selects is the smallest index of its own largest score (NaN
    skipped), exactly; and it equals the oracle's whenever the oracle's top-1 minus top-2
    exceeds twice the score tolerance (otherwise any list within the tolerance of the maximum).
Integer outputs compare bit for bit.
"""
from __future__ import annotations

from typing import Dict, Optional

import numpy as np
import torch

from paper_2603_02565_amd import flasheval as fe

RTOL = {"f32": 1e-4, "bf16": 2e-2}
SCORE_RTOL = {"f32": 1e-4, "bf16": 3e-2}


def rtol_for(cfg) -> float:
    return RTOL[cfg.dtype]


def normwise(gpu, ref) -> float:
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    scale = float(np.max(np.abs(ref))) if ref.size else 0.0
    err = float(np.max(np.abs(gpu - ref))) if ref.size else 0.0
    return err / scale if scale > 0 else err


def score_tol(cfg, scores_ref) -> float:
    """Absolute score tolerance of one request: SCORE_RTOL * max_k |s_ref[k]|."""
    ref = np.asarray(scores_ref, np.float64)
    ref = ref[~np.isnan(ref)]
    return SCORE_RTOL[cfg.dtype] * (float(np.max(np.abs(ref))) if ref.size else 0.0)


def min_argmax(s) -> int:
    """Smallest index of the largest non-NaN entry, -1 when every entry is NaN."""
    s = np.asarray(s, np.float64)
    ok = ~np.isnan(s)
    if not ok.any():
        return -1
    return int(np.flatnonzero(ok & (s == np.max(s[ok])))[0])


def check_selection(best_gpu: int, scores_ref: np.ndarray, tol: float) -> bool:
    """Selection parity against the oracle's scores: exact when the oracle's top-2 margin exceeds
    2*tol, else any list within tol of the maximum.  Returns whether the exact branch applied."""
    ref = np.asarray(scores_ref, np.float64)
    order = np.argsort(-ref, kind="stable")
    top = ref[order[0]]
    margin = top - ref[order[1]] if ref.size > 1 else np.inf
    if margin > 2 * tol:
        assert best_gpu == int(order[0]), (best_gpu, int(order[0]), margin, tol)
        return True
    assert 0 <= best_gpu < ref.size and ref[best_gpu] >= top - tol, (best_gpu, top, ref[best_gpu], tol)
    return False


def check_scores(cfg, scores_gpu, best_gpu: int, scores_ref, what="") -> Dict[str, float]:
    """Scores within the score tolerance, the selection of the GPU's own scores exact, and the
    selection against the oracle's scores.  Returns the measured error ratio
    max|ds| / max|s_ref| and whether the request was in the exact-selection regime."""
    g = np.asarray(scores_gpu, np.float64)
    ref = np.asarray(scores_ref, np.float64)
    tol = score_tol(cfg, ref)
    err = float(np.max(np.abs(g - ref)))
    scale = tol / SCORE_RTOL[cfg.dtype]
    assert err <= tol, (what, "scores", err / scale, SCORE_RTOL[cfg.dtype])
    assert int(best_gpu) == min_argmax(g), (what, "selection of the GPU's own scores", int(best_gpu), min_argmax(g))
    strict = check_selection(int(best_gpu), ref, tol)
    return {"ratio": err / scale if scale > 0 else err, "strict": strict}


def make_evaluator(cfg, W) -> fe.Evaluator:
    return fe.Evaluator(cfg.d, cfg.n_heads, cfg.n_layers, cfg.ffn, cfg.max_L, cfg.vocab, cfg.dtype, W,
                        attention=cfg.attention)


def upload(cfg, I: Dict) -> Dict[str, Optional[torch.Tensor]]:
    act = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    dev = torch.device("cuda", torch.cuda.current_device())
    out = {}
    for k in ("x", "pool"):
        out[k] = None if I.get(k) is None else torch.from_numpy(np.ascontiguousarray(I[k])).to(dev).to(act)
    out["ctx_ids"] = None if I.get("ctx_ids") is None else torch.from_numpy(
        np.ascontiguousarray(I["ctx_ids"], dtype=np.int32)).to(dev)
    out["lists"] = torch.from_numpy(np.ascontiguousarray(I["lists"], dtype=np.int32)).to(dev)
    return out


def fetch(bufs: Dict) -> Dict[str, np.ndarray]:
    torch.cuda.synchronize()
    res = {}
    for k in ("kv", "uniq", "n_uniq", "slot", "H", "seq", "Cp", "scores", "best"):
        t = bufs[k]
        res[k] = (t.float() if t.is_floating_point() else t).cpu().numpy()
    return res


def run_pass(cfg, W, I, ev: Optional[fe.Evaluator] = None) -> Dict[str, np.ndarray]:
    """Full pass of a generated workload; returns host copies of every output tensor."""
    own = ev is None
    if own:
        ev = make_evaluator(cfg, W)
    B, K, L = I["lists"].shape
    T = (I["x"] if I.get("x") is not None else I["ctx_ids"]).shape[1]
    ev.allocate(B, T, cfg.M, K, L)
    d = upload(cfg, I)
    bufs = ev.run(x=d["x"], ctx_ids=d["ctx_ids"], pool=d["pool"], lists=d["lists"])
    out = fetch(bufs)
    out["status"] = fe.fe_read_device_status(ev.handle, bufs["ws"], B)
    if own:
        ev.close()
    return out
