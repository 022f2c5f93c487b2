"""C ABI checks that need no GPU: the library loads, exports what the headers declare, and the
host-only entry points validate configurations.  No kernel is launched here."""
import ctypes
import os
import re

import numpy as np
import pytest

import gen
from paper_2603_02565_amd import flasheval as fe

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    for h in sorted(f for f in os.listdir(os.path.join(ROOT, "include")) if f.endswith(".h")):
        with open(os.path.join(ROOT, "include", h)) as f:
            text = re.sub(r"/\*.*?\*/", "", f.read(), flags=re.S)
        names |= set(re.findall(r"\b(fe_[a-z_]+)\s*\(", text))
    return names


def test_library_exports_every_declared_function():
    lib = fe.load_library()
    declared = _declared()
    assert {"fe_encode_context", "fe_encode_items", "fe_assemble", "fe_cross_sequence",
            "fe_score_select"} <= declared
    for name in declared:
        assert hasattr(lib, name), name
    assert declared == set(fe.EXPORTED)


def _cfg(c, **kw):
    f = fe.fe_config(c.d, c.n_heads, c.n_layers, c.ffn, c.max_L, c.vocab, fe.FE_BF16 if c.dtype == "bf16" else fe.FE_F32)
    for k, v in kw.items():
        setattr(f, k, v)
    return f


@pytest.mark.parametrize("cid", [0, 1, 3, 4])
def test_param_count_matches_generator(cid):
    c = gen.config(cid)
    W = gen.make_weights(c)
    assert fe.fe_param_count(_cfg(c)) == sum(v.size for v in W.values())
    assert sorted(fe.param_names(c.n_layers, c.vocab)) == sorted(W)
    flat = fe.pack_params(W, c.n_layers, c.vocab)
    assert flat.dtype == np.float32 and flat.size == fe.fe_param_count(_cfg(c))


@pytest.mark.parametrize("field,value,status", [
    ("d", 96, fe.FE_EUNSUPPORTED),          # width outside the supported set
    ("n_heads", 3, fe.FE_EINVAL),           # d not divisible by heads
    ("n_heads", 1, fe.FE_EUNSUPPORTED),     # head width 128
    ("n_layers", 0, fe.FE_EINVAL),
    ("n_layers", 9, fe.FE_EUNSUPPORTED),
    ("ffn_dim", 320, fe.FE_EUNSUPPORTED),   # not a multiple of 128 on a bf16 model
    ("max_L", 128, fe.FE_EUNSUPPORTED),
    ("dtype", 7, fe.FE_EINVAL),
    ("attention", 2, fe.FE_EINVAL),        # neither softmax nor linear
])
def test_config_validation(field, value, status):
    c = gen.config(1)
    with pytest.raises(fe.FeError) as e:
        fe.fe_param_count(_cfg(c, **{field: value}))
    assert e.value.status == status
    assert fe.load_library().fe_last_error().decode()


def test_bf16_needs_width_128():
    c = gen.config(0)
    with pytest.raises(fe.FeError) as e:
        fe.fe_param_count(_cfg(c, dtype=fe.FE_BF16))
    assert e.value.status == fe.FE_EUNSUPPORTED


def test_null_config_is_einval():
    n = ctypes.c_size_t()
    assert fe.load_library().fe_param_count(None, ctypes.byref(n)) == fe.FE_EINVAL


def test_trace_toggle_without_launches():
    fe.fe_trace_enable(True)
    out = fe.fe_trace_read()
    fe.fe_trace_enable(False)
    assert set(out) == {"gemm", "attention", "layernorm", "dedup", "gather", "assemble", "score_select", "fill", "ffn",
                        "layer", "post", "linear"}
    assert all(v == (0.0, 0) for v in out.values())


def test_trace_launch_records_without_launches():
    fe.fe_trace_enable(True)
    assert fe.fe_trace_read_launches() == []
    fe.fe_trace_enable(False)


def _train_cfg(c, **kw):
    f = fe.fe_config(c.d, c.n_heads, c.n_layers, c.ffn, c.max_L, c.vocab, fe.FE_F32, fe.FE_ATTN_SOFTMAX)
    for k, v in kw.items():
        setattr(f, k, v)
    return f


def test_train_workspace_grows_with_the_batch():
    c = gen.config(1)
    small = fe.fe_train_workspace_size(_train_cfg(c), 2, 64, 200, 50, 10)
    big = fe.fe_train_workspace_size(_train_cfg(c), 4, 64, 200, 50, 10)
    longer = fe.fe_train_workspace_size(_train_cfg(c), 2, 128, 200, 50, 10)
    assert 0 < small < big and small < longer and small % 256 == 0


@pytest.mark.parametrize("kw,dims,status", [
    (dict(dtype=fe.FE_BF16), (2, 64, 200, 50, 10), fe.FE_EUNSUPPORTED),           # fp32 models only
    (dict(attention=fe.FE_ATTN_LINEAR), (2, 64, 200, 50, 10), fe.FE_EUNSUPPORTED),
    ({}, (2, 64, 200, 1025, 10), fe.FE_EUNSUPPORTED),                              # K > 1024
    ({}, (2, 64, 200, 50, 11), fe.FE_EINVAL),                                      # L > max_L
    ({}, (0, 64, 200, 50, 10), fe.FE_EINVAL),
    (dict(vocab=40), (2, 64, 200, 50, 10), fe.FE_EINVAL),                          # token ids need M = vocab
    ({}, (2_000_000, 64, 200, 50, 10), fe.FE_EUNSUPPORTED),                       # rows past 32-bit row indexing
])
def test_train_validation(kw, dims, status):
    c = gen.config(1)
    with pytest.raises(fe.FeError) as e:
        fe.fe_train_workspace_size(_train_cfg(c, **kw), *dims)
    assert e.value.status == status
    assert fe.load_library().fe_last_error().decode()


def test_train_binding_rejects_wrong_dtype_before_any_call():
    """The binding hands raw pointers to the library; a float64 loss buffer (say, under a float64
    default dtype) would be half-written, so it is refused before the call."""
    import torch
    c = gen.config(0)
    cfg = _train_cfg(c)
    n = fe.fe_param_count(cfg)
    P = torch.zeros(n, dtype=torch.float32)
    with pytest.raises(ValueError, match="loss"):
        fe.fe_train_grads(cfg, P, 1, c.T, c.M, c.K, c.L, None, None, None, None, None, fe.FE_LOSS_CE,
                          torch.zeros(1, dtype=torch.float64), None, torch.zeros_like(P), torch.zeros(8, dtype=torch.uint8))
    with pytest.raises(ValueError, match="grads"):
        fe.fe_train_grads(cfg, P, 1, c.T, c.M, c.K, c.L, None, None, None, None, None, fe.FE_LOSS_CE,
                          torch.zeros(1), None, torch.zeros(n - 1), torch.zeros(8, dtype=torch.uint8))


def _train_call(cfg, c, *, loss_kind=fe.FE_LOSS_CE, ws=1 << 20, ws_bytes=None, pool=8192, x=8192):
    """fe_train_grads with placeholder device addresses: every case below is refused by the host-side
    checks before anything touches them."""
    n = fe.fe_param_count(cfg)
    need = fe.fe_train_workspace_size(cfg, 1, c.T, c.M, c.K, c.L)
    lib = fe.load_library()
    return lib.fe_train_grads(ctypes.byref(cfg), 4096, 1, c.T, c.M, c.K, c.L, x, None, pool, 12288, 16384, loss_kind,
                              20480, None, 24576, ws, need if ws_bytes is None else ws_bytes, None), need


@pytest.mark.parametrize("case", ["loss_kind", "misaligned", "small", "no_pool"])
def test_train_grads_host_checks(case):
    c = gen.config(0)
    cfg = _train_cfg(c)
    if case == "loss_kind":
        st, _ = _train_call(cfg, c, loss_kind=3)
    elif case == "misaligned":
        st, _ = _train_call(cfg, c, ws=(1 << 20) + 64)
    elif case == "small":
        st, need = _train_call(cfg, c, ws_bytes=1024)
    else:
        st, _ = _train_call(cfg, c, pool=None)
    assert st == fe.FE_EINVAL
    msg = fe.load_library().fe_last_error().decode()
    assert {"loss_kind": "loss_kind", "misaligned": "aligned", "small": "workspace", "no_pool": "pool"}[case] in msg


def test_executor_host_checks():
    """The executor's entry points reject NULL handles and arguments before touching the device."""
    lib = fe.load_library()
    out = ctypes.c_void_p()
    assert lib.fe_executor_create(None, 2, ctypes.byref(out)) == fe.FE_EINVAL
    assert lib.fe_executor_submit(None, None, None) == fe.FE_EINVAL
    assert lib.fe_executor_join(None, None) == fe.FE_EINVAL
    lib.fe_executor_destroy(None)
