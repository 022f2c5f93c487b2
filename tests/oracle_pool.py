"""Stage-by-stage comparison of a whole batch with the cached-order float64 oracle, one request
per task in a pool of CPU worker processes.

Test infrastructure: the workers are started with the "spawn" method and import only numpy,
`gen` and `oracle` (never torch or the HIP library); each regenerates the workload's inputs and
weights from its seeded configuration and compares the GPU's outputs of one request with the
oracle's (`oracle.evaluate_cached`, which the CPU tests pin to the candidate-factorised
`oracle.evaluate_naive`).  Every request of a batch is covered, at the cost of the oracle's CPU
time spread over up to 16 processes.
"""
from __future__ import annotations

import multiprocessing as mp
import os
from typing import Dict, List, Optional

import numpy as np

_POOL = None
_CACHE: Dict = {}


def _workload(cfg):
    import gen
    if cfg not in _CACHE:
        _CACHE.clear()
        _CACHE[cfg] = (gen.make_weights(cfg), gen.make_inputs(cfg))
    return _CACHE[cfg]


def _normwise(gpu, ref) -> float:
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    if not ref.size:
        return 0.0
    scale = float(np.max(np.abs(ref)))
    err = float(np.max(np.abs(gpu - ref)))
    return err / scale if scale > 0 else err


def compare_request(job) -> Dict:
    """One request: the oracle's stages and the GPU's, reduced to error ratios and exact flags."""
    import oracle
    cfg, b, g = job
    W, I = _workload(cfg)
    r = oracle.evaluate_cached(cfg, W, I, requests=[b], stages=True)[b]
    out = {"b": b}
    if g.get("kv") is not None:
        if cfg.attention == "linear":
            out["kv"] = [_normwise(g["kv"][l], oracle.linear_kv_state(r["kv"][l][0], r["kv"][l][1], cfg.n_heads))
                         for l in range(cfg.n_layers)]
        else:
            out["kv"] = [max(_normwise(g["kv"][l][0], r["kv"][l][0]), _normwise(g["kv"][l][1], r["kv"][l][1]))
                         for l in range(cfg.n_layers)]
    U = len(r["uniq"])
    out["U"] = U
    out["n_uniq_ok"] = int(g["n_uniq"]) == U
    out["uniq_ok"] = bool(np.array_equal(g["uniq"][:U], r["uniq"]) and np.all(g["uniq"][U:] == -1))
    out["slot_ok"] = bool(np.array_equal(g["slot"], r["slot"]))
    out["H"] = _normwise(g["H"][:U], r["H"])
    out["H_pad_zero"] = bool(np.all(g["H"][U:] == 0))
    out["seq"] = _normwise(g["seq"], r["seq"])
    out["Cp"] = _normwise(g["Cp"], r["Cp"])
    out["scores_ref"] = np.asarray(r["scores"], np.float64)
    out["best_ref"] = int(r["best"])
    return out


def pool_size() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _pool():
    global _POOL
    if _POOL is None:
        saved = {k: os.environ.get(k) for k in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS")}
        for k in saved:
            os.environ[k] = "1"          # one BLAS thread per worker; the workers themselves are the parallelism
        try:
            _POOL = mp.get_context("spawn").Pool(pool_size())
        finally:
            for k, v in saved.items():
                if v is None:
                    os.environ.pop(k, None)
                else:
                    os.environ[k] = v
    return _POOL


def compare_batch(cfg, out: Dict[str, np.ndarray], requests: Optional[List[int]] = None) -> List[Dict]:
    """compare_request for every request of `out` (a `run_pass` result of the generated workload
    `cfg`), in request order."""
    reqs = list(range(cfg.B)) if requests is None else list(requests)
    jobs = []
    for b in reqs:
        g = {k: out[k][b] for k in ("uniq", "n_uniq", "slot", "H", "seq", "Cp")}
        if out.get("kv") is None:
            g["kv"] = None
        elif cfg.attention == "linear":           # [n][B][H][dh+1][dh]
            g["kv"] = np.ascontiguousarray(out["kv"][:, b])
        else:                                     # [n][2][B][T][d]
            g["kv"] = np.ascontiguousarray(out["kv"][:, :, b])
        jobs.append((cfg, b, g))
    return _pool().map(compare_request, jobs, chunksize=1)


def close() -> None:
    global _POOL
    if _POOL is not None:
        _POOL.close()
        _POOL.join()
        _POOL = None
