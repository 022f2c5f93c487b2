"""Python binding of libflasheval (ctypes).  Argument marshalling only: every step of the pass
runs in the library's HIP kernels.  Functions carry the names of the C ABI in
include/flasheval.h and take torch tensors that live on the current HIP device; the stream is
torch's current stream unless one is given.

There is no fallback: if libflasheval.so has not been built, `load_library` raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libflasheval.so")

FE_OK, FE_EINVAL, FE_EUNSUPPORTED, FE_ENOMEM, FE_EHIP = range(5)
FE_F32, FE_BF16 = 0, 1
FE_ATTN_SOFTMAX, FE_ATTN_LINEAR = 0, 1
FE_DEV_BAD_INDEX, FE_DEV_BAD_TOKEN = 1, 2
FE_LOSS_MSE, FE_LOSS_BCE, FE_LOSS_CE = 0, 1, 2
LOSS_KIND = {"mse": FE_LOSS_MSE, "bce": FE_LOSS_BCE, "ce": FE_LOSS_CE}

EXPORTED = ("fe_param_count", "fe_model_create", "fe_model_destroy", "fe_workspace_size", "fe_kv_size", "fe_last_error",
            "fe_read_device_status", "fe_encode_context", "fe_encode_items", "fe_assemble", "fe_cross_sequence",
            "fe_cross_sequence_noalloc", "fe_score_select", "fe_encode_sequences", "fe_score_objectives", "fe_naive_workspace_size", "fe_evaluate_naive", "fe_trace_enable", "fe_trace_read",
            "fe_trace_read_launches", "fe_trace_family", "fe_train_workspace_size", "fe_train_grads",
            "fe_executor_create", "fe_executor_submit", "fe_executor_join", "fe_executor_destroy")
FE_EXECUTOR_MAX_STREAMS = 8
FE_TRACE_FAMILIES = 12


class FeError(RuntimeError):
    def __init__(self, status: int, where: str, msg: str):
        super().__init__(f"{where} -> status {status}: {msg}")
        self.status = status


class fe_config(ctypes.Structure):
    _fields_ = [("d", ctypes.c_int32), ("n_heads", ctypes.c_int32), ("n_layers", ctypes.c_int32),
                ("ffn_dim", ctypes.c_int32), ("max_L", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("attention", ctypes.c_int32)]


class fe_pass_args(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("T", ctypes.c_int32), ("M", ctypes.c_int32), ("K", ctypes.c_int32),
                ("L", ctypes.c_int32), ("x", ctypes.c_void_p), ("ctx_ids", ctypes.c_void_p), ("pool", ctypes.c_void_p),
                ("lists", ctypes.c_void_p), ("kv", ctypes.c_void_p), ("uniq", ctypes.c_void_p),
                ("n_uniq", ctypes.c_void_p), ("slot", ctypes.c_void_p), ("H", ctypes.c_void_p), ("seq", ctypes.c_void_p),
                ("Cp", ctypes.c_void_p), ("scores", ctypes.c_void_p), ("best", ctypes.c_void_p), ("ws", ctypes.c_void_p),
                ("ws_bytes", ctypes.c_size_t)]


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libflasheval.so (once).  Raises if it is missing: build it with __graft_entry__.build()."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing; build the HIP library first (python -c "
                           "'import __graft_entry__ as g; g.build()')")
    lib = ctypes.CDLL(path)
    P, I, Z, S = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t, ctypes.c_int
    cfgp = ctypes.POINTER(fe_config)
    sig = {
        "fe_param_count": (S, [cfgp, ctypes.POINTER(Z)]),
        "fe_model_create": (S, [cfgp, P, Z, ctypes.POINTER(P)]),
        "fe_model_destroy": (None, [P]),
        "fe_workspace_size": (S, [P, I, I, I, I, I, ctypes.POINTER(Z)]),
        "fe_kv_size": (S, [P, I, I, ctypes.POINTER(Z)]),
        "fe_last_error": (ctypes.c_char_p, []),
        "fe_read_device_status": (S, [P, P, I, P, P]),
        "fe_encode_context": (S, [P, I, I, P, P, P, P, Z, P]),
        "fe_encode_items": (S, [P, I, I, P, P, I, I, P, I, P, P, P, P, P, Z, P]),
        "fe_assemble": (S, [P, I, I, I, I, P, P, P, P]),
        "fe_cross_sequence": (S, [P, I, I, I, P, P, P, Z, P]),
        "fe_cross_sequence_noalloc": (S, [P, I, I, I, P, P, P]),
        "fe_score_select": (S, [P, I, I, P, P, P, P]),
        "fe_encode_sequences": (S, [P, I, I, I, P, P, P, Z, P]),
        "fe_score_objectives": (S, [P, I, I, P, I, P, P, P, P, P, P, P]),
        "fe_naive_workspace_size": (S, [P, I, I, I, I, I, I, ctypes.POINTER(Z)]),
        "fe_evaluate_naive": (S, [P, I, I, I, I, I, P, P, P, P, P, P, P, P, Z, P]),
        "fe_trace_enable": (S, [I]),
        "fe_trace_read": (S, [P, P]),
        "fe_trace_read_launches": (S, [P, P, ctypes.c_int64, P]),
        "fe_trace_family": (ctypes.c_char_p, [I]),
        "fe_train_workspace_size": (S, [cfgp, I, I, I, I, I, ctypes.POINTER(Z)]),
        "fe_train_grads": (S, [cfgp, P, I, I, I, I, I, P, P, P, P, P, I, P, P, P, P, Z, P]),
        "fe_executor_create": (S, [P, I, ctypes.POINTER(P)]),
        "fe_executor_submit": (S, [P, ctypes.POINTER(fe_pass_args), P]),
        "fe_executor_join": (S, [P, P]),
        "fe_executor_destroy": (None, [P]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def _check(status: int, where: str) -> None:
    if status != FE_OK:
        raise FeError(status, where, load_library().fe_last_error().decode())


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    import torch
    return torch.cuda.current_stream().cuda_stream


# ---------------------------------------------------------------------------------------------
# Parameter order of fe_model_create (as documented in include/flasheval.h)
# ---------------------------------------------------------------------------------------------

_ENC = ("ln1.g", "ln1.b", "wqkv", "bqkv", "wo", "bo", "ln2.g", "ln2.b", "w1", "b1", "w2", "b2")
_ITEM = ("ln1.g", "ln1.b", "wqkv", "bqkv", "wo", "bo", "ln2.g", "ln2.b", "wq", "bq", "wo2", "bo2",
         "ln3.g", "ln3.b", "w1", "b1", "w2", "b2")


def param_names(n_layers: int, vocab: int) -> List[str]:
    names: List[str] = []
    names += [f"ctx.{l}.{p}" for l in range(n_layers) for p in _ENC]
    names += ["ctx.lnf.g", "ctx.lnf.b"]
    names += [f"ctx.kv.{l}.{p}" for l in range(n_layers) for p in ("wk", "bk", "wv", "bv")]
    names += [f"item.{l}.{p}" for l in range(n_layers) for p in _ITEM]
    names += ["item.lnf.g", "item.lnf.b"]
    names += [f"seq.{l}.{p}" for l in range(n_layers) for p in _ENC]
    names += ["seq.lnf.g", "seq.lnf.b"]
    names += [f"cross.{l}.{p}" for l in range(n_layers) for p in _ENC]
    names += ["cross.lnf.g", "cross.lnf.b"]
    names += ["cls", "pos", "head.w", "head.b"]
    if vocab:
        names.append("emb")
    return names


def pack_params(params: Dict[str, np.ndarray], n_layers: int, vocab: int) -> np.ndarray:
    """Flat float32 array of every parameter in fe_model_create order."""
    return np.concatenate([np.ascontiguousarray(params[n], dtype=np.float32).reshape(-1)
                           for n in param_names(n_layers, vocab)])


# ---------------------------------------------------------------------------------------------
# C functions (same names as the ABI)
# ---------------------------------------------------------------------------------------------

def fe_param_count(cfg: fe_config) -> int:
    n = ctypes.c_size_t()
    _check(load_library().fe_param_count(ctypes.byref(cfg), ctypes.byref(n)), "fe_param_count")
    return n.value


def fe_model_create(cfg: fe_config, flat: np.ndarray) -> int:
    flat = np.ascontiguousarray(flat, dtype=np.float32)
    h = ctypes.c_void_p()
    _check(load_library().fe_model_create(ctypes.byref(cfg), flat.ctypes.data, flat.size, ctypes.byref(h)),
           "fe_model_create")
    return h.value


def fe_model_destroy(model: int) -> None:
    load_library().fe_model_destroy(model)


def fe_workspace_size(model: int, B: int, T: int, M: int, K: int, L: int) -> int:
    n = ctypes.c_size_t()
    _check(load_library().fe_workspace_size(model, B, T, M, K, L, ctypes.byref(n)), "fe_workspace_size")
    return n.value


def fe_kv_size(model: int, B: int, T: int) -> int:
    n = ctypes.c_size_t()
    _check(load_library().fe_kv_size(model, B, T, ctypes.byref(n)), "fe_kv_size")
    return n.value


def fe_read_device_status(model: int, ws, B: int, stream=None) -> np.ndarray:
    out = np.zeros(B, dtype=np.int32)
    _check(load_library().fe_read_device_status(model, _ptr(ws), B, _stream(stream), out.ctypes.data),
           "fe_read_device_status")
    return out


def fe_encode_context(model: int, B: int, T: int, x, ctx_ids, kv, ws, stream=None) -> None:
    _check(load_library().fe_encode_context(model, B, T, _ptr(x), _ptr(ctx_ids), _ptr(kv), _ptr(ws),
                                            ws.numel() * ws.element_size(), _stream(stream)), "fe_encode_context")


def fe_encode_items(model: int, B: int, M: int, pool, lists, K: int, L: int, kv, T: int, uniq, n_uniq, slot, H, ws,
                    stream=None) -> None:
    _check(load_library().fe_encode_items(model, B, M, _ptr(pool), _ptr(lists), K, L, _ptr(kv), T, _ptr(uniq),
                                          _ptr(n_uniq), _ptr(slot), _ptr(H), _ptr(ws),
                                          ws.numel() * ws.element_size(), _stream(stream)), "fe_encode_items")


def fe_assemble(model: int, B: int, K: int, L: int, U_cap: int, slot, H, seq, stream=None) -> None:
    _check(load_library().fe_assemble(model, B, K, L, U_cap, _ptr(slot), _ptr(H), _ptr(seq), _stream(stream)),
           "fe_assemble")


def fe_cross_sequence(model: int, B: int, K: int, L: int, seq, Cp, ws, stream=None) -> None:
    _check(load_library().fe_cross_sequence(model, B, K, L, _ptr(seq), _ptr(Cp), _ptr(ws),
                                            ws.numel() * ws.element_size(), _stream(stream)), "fe_cross_sequence")


FE_NOALLOC_SCRATCH_BYTES = 32 << 20


def fe_executor_create(model: int, n_streams: int) -> int:
    out = ctypes.c_void_p()
    _check(load_library().fe_executor_create(model, n_streams, ctypes.byref(out)), "fe_executor_create")
    return out.value


def fe_executor_submit(ex: int, B: int, T: int, M: int, K: int, L: int, x, ctx_ids, pool, lists, kv, uniq, n_uniq,
                       slot, H, seq, Cp, scores, best, ws, stream=None) -> None:
    a = fe_pass_args(B, T, M, K, L, _ptr(x), _ptr(ctx_ids), _ptr(pool), _ptr(lists), _ptr(kv), _ptr(uniq),
                     _ptr(n_uniq), _ptr(slot), _ptr(H), _ptr(seq), _ptr(Cp), _ptr(scores), _ptr(best), _ptr(ws),
                     ws.numel() * ws.element_size())
    _check(load_library().fe_executor_submit(ex, ctypes.byref(a), _stream(stream)), "fe_executor_submit")


def fe_executor_join(ex: int, stream=None) -> None:
    _check(load_library().fe_executor_join(ex, _stream(stream)), "fe_executor_join")


def fe_executor_destroy(ex: int) -> None:
    load_library().fe_executor_destroy(ex)


def fe_cross_sequence_noalloc(model: int, B: int, K: int, L: int, seq, Cp, stream=None) -> None:
    """fe_cross_sequence with the library's static scratch instead of a workspace (allocates nothing)."""
    _check(load_library().fe_cross_sequence_noalloc(model, B, K, L, _ptr(seq), _ptr(Cp), _stream(stream)),
           "fe_cross_sequence_noalloc")


def fe_score_select(model: int, B: int, K: int, Cp, scores, best, stream=None) -> None:
    _check(load_library().fe_score_select(model, B, K, _ptr(Cp), _ptr(scores), _ptr(best), _stream(stream)),
           "fe_score_select")


def fe_encode_sequences(model: int, B: int, K: int, L: int, seq, C, ws, stream=None) -> None:
    _check(load_library().fe_encode_sequences(model, B, K, L, _ptr(seq), _ptr(C), _ptr(ws),
                                              ws.numel() * ws.element_size(), _stream(stream)), "fe_encode_sequences")


def fe_score_objectives(model: int, B: int, K: int, Cp, n_obj: int, head_w, head_b, fuse_w, obj_scores, scores, best,
                        stream=None) -> None:
    _check(load_library().fe_score_objectives(model, B, K, _ptr(Cp), n_obj, _ptr(head_w), _ptr(head_b), _ptr(fuse_w),
                                              _ptr(obj_scores), _ptr(scores), _ptr(best), _stream(stream)),
           "fe_score_objectives")


def fe_naive_workspace_size(model: int, B: int, T: int, M: int, K: int, L: int, token_ids: bool) -> int:
    n = ctypes.c_size_t()
    _check(load_library().fe_naive_workspace_size(model, B, T, M, K, L, 1 if token_ids else 0, ctypes.byref(n)),
           "fe_naive_workspace_size")
    return n.value


def fe_evaluate_naive(model: int, B: int, T: int, M: int, K: int, L: int, x, ctx_ids, pool, lists, Cp, scores, best,
                      ws, stream=None) -> None:
    _check(load_library().fe_evaluate_naive(model, B, T, M, K, L, _ptr(x), _ptr(ctx_ids), _ptr(pool), _ptr(lists),
                                            _ptr(Cp), _ptr(scores), _ptr(best), _ptr(ws),
                                            ws.numel() * ws.element_size(), _stream(stream)), "fe_evaluate_naive")


def fe_train_workspace_size(cfg: fe_config, B: int, T: int, M: int, K: int, L: int) -> int:
    n = ctypes.c_size_t()
    _check(load_library().fe_train_workspace_size(ctypes.byref(cfg), B, T, M, K, L, ctypes.byref(n)),
           "fe_train_workspace_size")
    return n.value


def _need(t, name: str, dtype, numel: int) -> None:
    """Argument check for tensors handed to the library as raw pointers: dtype, size, contiguity."""
    if t is None or isinstance(t, int):
        return
    if t.dtype != dtype or t.numel() != numel or not t.is_contiguous():
        raise ValueError(f"{name}: expected a contiguous {dtype} tensor of {numel} elements, got {t.dtype} "
                         f"{tuple(t.shape)}")


def fe_train_grads(cfg: fe_config, params, B: int, T: int, M: int, K: int, L: int, x, ctx_ids, pool, lists, relevant,
                   loss_kind: int, loss, scores, grads, ws, stream=None) -> None:
    import torch
    n = fe_param_count(cfg)
    _need(params, "params", torch.float32, n)
    _need(grads, "grads", torch.float32, n)
    _need(loss, "loss", torch.float32, 1)
    _need(scores, "scores", torch.float32, B * K)
    _need(x, "x", torch.float32, B * T * cfg.d)
    _need(pool, "pool", torch.float32, B * M * cfg.d)
    _need(ctx_ids, "ctx_ids", torch.int32, B * T)
    _need(lists, "lists", torch.int32, B * K * L)
    _need(relevant, "relevant", torch.int32, B * M)
    _check(load_library().fe_train_grads(ctypes.byref(cfg), _ptr(params), B, T, M, K, L, _ptr(x), _ptr(ctx_ids),
                                         _ptr(pool), _ptr(lists), _ptr(relevant), loss_kind, _ptr(loss), _ptr(scores),
                                         _ptr(grads), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)),
           "fe_train_grads")


def fe_trace_enable(on: bool) -> None:
    _check(load_library().fe_trace_enable(1 if on else 0), "fe_trace_enable")


def fe_trace_read_launches(capacity: int = 1 << 16) -> List[Tuple[str, float]]:
    """Recorded launches in enqueue order: (family name, kernel ms) each; consumes the records."""
    lib = load_library()
    fam = np.zeros(capacity, dtype=np.int32)
    ms = np.zeros(capacity, dtype=np.float64)
    n = ctypes.c_int64(0)
    _check(lib.fe_trace_read_launches(fam.ctypes.data, ms.ctypes.data, capacity, ctypes.byref(n)),
           "fe_trace_read_launches")
    return [(lib.fe_trace_family(int(fam[i])).decode(), float(ms[i])) for i in range(n.value)]


def fe_trace_read() -> Dict[str, Tuple[float, int]]:
    """{family: (summed kernel ms, launches)} since the last read; synchronises the traced events."""
    ms = np.zeros(FE_TRACE_FAMILIES, dtype=np.float64)
    n = np.zeros(FE_TRACE_FAMILIES, dtype=np.int64)
    lib = load_library()
    _check(lib.fe_trace_read(ms.ctypes.data, n.ctypes.data), "fe_trace_read")
    return {lib.fe_trace_family(i).decode(): (float(ms[i]), int(n[i])) for i in range(FE_TRACE_FAMILIES)}


# ---------------------------------------------------------------------------------------------
# Convenience: one model plus the buffers of one batch shape
# ---------------------------------------------------------------------------------------------

class Evaluator:
    """Owns a model handle and, per batch shape, the device buffers of the five calls.

    `params` maps the parameter names of `param_names` to float arrays; `dtype` is "f32" or
    "bf16".  All tensors are allocated with torch on the current device.
    """

    def __init__(self, d: int, n_heads: int, n_layers: int, ffn_dim: int, max_L: int, vocab: int, dtype: str,
                 params: Dict[str, np.ndarray], attention: str = "softmax"):
        import torch
        if not torch.cuda.is_available():
            raise RuntimeError("Evaluator needs a HIP device")
        if attention not in ("softmax", "linear"):
            raise ValueError(f"attention must be 'softmax' or 'linear', got {attention!r}")
        self.cfg = fe_config(d, n_heads, n_layers, ffn_dim, max_L, vocab, FE_BF16 if dtype == "bf16" else FE_F32,
                             FE_ATTN_LINEAR if attention == "linear" else FE_ATTN_SOFTMAX)
        self.d, self.n_layers, self.vocab, self.n_heads = d, n_layers, vocab, n_heads
        self.attention = attention
        self.act = torch.bfloat16 if dtype == "bf16" else torch.float32
        self.handle = fe_model_create(self.cfg, pack_params(params, n_layers, vocab))
        self.buffers = None
        self.naive_buffers = None

    def close(self) -> None:
        if self.handle:
            fe_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def allocate(self, B: int, T: int, M: int, K: int, L: int) -> Dict:
        import torch
        dev = torch.device("cuda", torch.cuda.current_device())
        d, n = self.d, self.n_layers
        U_cap = min(M, K * L)
        ws_bytes = fe_workspace_size(self.handle, B, T, M, K, L)
        i32 = torch.int32
        self.buffers = dict(
            shape=(B, T, M, K, L), U_cap=U_cap,
            kv=self._kv_tensor(B, T, dev),
            uniq=torch.empty((B, U_cap), dtype=i32, device=dev),
            n_uniq=torch.empty((B,), dtype=i32, device=dev),
            slot=torch.empty((B, K, L), dtype=i32, device=dev),
            H=torch.empty((B, U_cap, d), dtype=self.act, device=dev),
            seq=torch.empty((B, K, L + 1, d), dtype=self.act, device=dev),
            Cp=torch.empty((B, K, d), dtype=torch.float32, device=dev),
            scores=torch.empty((B, K), dtype=torch.float32, device=dev),
            best=torch.empty((B,), dtype=i32, device=dev),
            ws=torch.empty((ws_bytes,), dtype=torch.uint8, device=dev),
        )
        return self.buffers

    def _kv_tensor(self, B: int, T: int, dev):
        """fe_encode_context's output: keys/values [n][2][B][T][d] act, or on linear-attention
        models the per-head state [n][B][H][dh+1][dh] fp32 (fe_kv_size bytes either way)."""
        import torch
        n, d, H = self.n_layers, self.d, self.n_heads
        if self.attention == "linear":
            shape, dt = (n, B, H, d // H + 1, d // H), torch.float32
        else:
            shape, dt = (n, 2, B, T, d), self.act
        t = torch.empty(shape, dtype=dt, device=dev)
        assert t.numel() * t.element_size() == fe_kv_size(self.handle, B, T)
        return t

    def run(self, x=None, ctx_ids=None, pool=None, lists=None, stream=None, buffers=None) -> Dict:
        """Enqueue the five calls on device tensors already resident on the GPU (into `buffers`, a
        dict from `allocate`, else the last allocated set)."""
        b = self.buffers if buffers is None else buffers
        B, T, M, K, L = b["shape"]
        h = self.handle
        fe_encode_context(h, B, T, x, ctx_ids, b["kv"], b["ws"], stream)
        fe_encode_items(h, B, M, pool, lists, K, L, b["kv"], T, b["uniq"], b["n_uniq"], b["slot"], b["H"], b["ws"],
                        stream)
        fe_assemble(h, B, K, L, b["U_cap"], b["slot"], b["H"], b["seq"], stream)
        fe_cross_sequence(h, B, K, L, b["seq"], b["Cp"], b["ws"], stream)
        fe_score_select(h, B, K, b["Cp"], b["scores"], b["best"], stream)
        return b

    def allocate_naive(self, B: int, T: int, M: int, K: int, L: int, token_ids: bool) -> Dict:
        """Outputs and workspace of the candidate-factorised baseline (fe_evaluate_naive)."""
        import torch
        dev = torch.device("cuda", torch.cuda.current_device())
        ws_bytes = fe_naive_workspace_size(self.handle, B, T, M, K, L, token_ids)
        self.naive_buffers = dict(
            shape=(B, T, M, K, L),
            Cp=torch.empty((B, K, self.d), dtype=torch.float32, device=dev),
            scores=torch.empty((B, K), dtype=torch.float32, device=dev),
            best=torch.empty((B,), dtype=torch.int32, device=dev),
            ws=torch.empty((ws_bytes,), dtype=torch.uint8, device=dev),
        )
        return self.naive_buffers

    def run_naive(self, x=None, ctx_ids=None, pool=None, lists=None, stream=None) -> Dict:
        """Enqueue the candidate-factorised evaluator (no reuse) on resident device tensors."""
        b = self.naive_buffers
        B, T, M, K, L = b["shape"]
        fe_evaluate_naive(self.handle, B, T, M, K, L, x, ctx_ids, pool, lists, b["Cp"], b["scores"], b["best"],
                          b["ws"], stream)
        return b


class Executor:
    """Whole passes of independent batches, round-robin over `n_streams` HIP streams of the
    library (fe_executor_*).  Give every stream its own buffer set (`Evaluator.allocate`): pass i
    writes set i mod n_streams, so a set is reused only after n_streams - 1 other passes."""

    def __init__(self, evaluator: "Evaluator", n_streams: int):
        self.evaluator = evaluator
        self.n_streams = n_streams
        self.handle = fe_executor_create(evaluator.handle, n_streams)

    def submit(self, buffers: Dict, x=None, ctx_ids=None, pool=None, lists=None, stream=None) -> Dict:
        """Enqueue one pass into `buffers` after the work already on `stream` (the inputs')."""
        b = buffers
        B, T, M, K, L = b["shape"]
        fe_executor_submit(self.handle, B, T, M, K, L, x, ctx_ids, pool, lists, b["kv"], b["uniq"], b["n_uniq"],
                           b["slot"], b["H"], b["seq"], b["Cp"], b["scores"], b["best"], b["ws"], stream)
        return b

    def join(self, stream=None) -> None:
        """Make `stream` wait for every submitted pass."""
        fe_executor_join(self.handle, stream)

    def close(self) -> None:
        if self.handle:
            fe_executor_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
