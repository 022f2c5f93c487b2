#!/usr/bin/env python3
"""Throughput of the joint-evaluation forward pass on one MI355X.

A step is one pass of all five C-ABI calls (context encoding, distinct-item encoding, assembly,
sequence + cross-sequence encoding, scoring + argmax) over one batch of synthetic requests whose
inputs are already resident in HBM.  The default workload is the RecSys base batch (B=64
requests, T=256 context rows, d=128, 4 heads, 2 layers per module, pool M=200, K=50 lists of
L=10); `--workload 2 --K k` runs the K sweep on the same shapes.

Prints one JSON line:  lists/s over the timed steps, p50/p90 step latency, the roofline of the
dominant kernel family (from HIP events around each launch in a second, traced pass over the
same steps), per-family kernel times, MFMA utilisation of the matrix-product stages, the HBM
fraction of the assembly kernel, and the CPU oracle timed on a bounded sample on this host.
"""
from __future__ import annotations

import argparse
import json
from dataclasses import replace
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "candidate lists scored/sec at K=50 (B=64,L=10); MFMA util %; p50 latency"
PEAK_BF16_TFLOPS = 256 * 4096 * 2.4e9 / 1e12     # dense bf16 matrix-core peak, 2516.6 TFLOP/s
PEAK_FP32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0
ASM_REPS = 100           # assembly launches per captured graph (gather-stage timing)
PIPE_STREAMS = 3         # batches in flight in the pipelined executor (one buffer set each)


def assemble_bytes(c, U):
    """Algorithmic HBM bytes of the assembly: write every [CLS; items] row once, read each
    distinct encoding once, read the slot indices."""
    d, B, K, S = c.d, c.B, c.K, c.L + 1
    esz = 2 if c.dtype == "bf16" else 4
    return B * K * S * d * esz + sum(U) * d * esz + B * K * c.L * 4


def module_parts(d, F, n, rows, groups, S, first_row_only=False):
    """Algorithmic flops of an encoder module of n pre-LN blocks over `groups` groups of S rows,
    split into (q|k|v projections, attention, output projection + FFN).

    Per row and block: q|k|v 6 d^2, output projection 2 d^2, FFN 4 d F; per group and block:
    attention 4 S^2 d (Q K^T and P V).  When only the first row of each group leaves the module
    (the [CLS] rows of the sequence encoder), the last block needs keys and values of every row
    but the query, the attention, the output projection and the FFN of the first rows alone.
    """
    proj = n * 6.0 * d * d * rows
    attn = n * 4.0 * S * S * d * groups
    tail = n * (2.0 * d * d + 4.0 * d * F) * rows
    if first_row_only:
        proj -= 2.0 * d * d * (rows - groups)
        attn -= 4.0 * S * d * (S - 1) * groups
        tail -= (2.0 * d * d + 4.0 * d * F) * (rows - groups)
    return proj, attn, tail


def family_flops(c, U, fam_names):
    """Split the algorithmic flops of one pass over the kernel families that ran.

    Fused kernels take the work of the stages they contain: "layer" (a whole module of short
    groups in one kernel: the sequence encoder, and the cross-sequence and context modules when
    their groups are short), "post" (output projection and FFN, or query projection, after a
    separate attention kernel, and the key/value cache in the last context tail), "attention"
    (with the q|k|v projection when the fused self-attention kernel applies), "gemm" (separate
    projections), "linear" (linear attention: per head the state sum_t phi(k_t) v_t^T, 2 dh^2
    flops per key, and its application, 2 dh (dh + 1) per query).
    """
    d, F, n, B, T, K, S = c.d, c.ffn, c.n_layers, c.B, c.T, c.K, c.L + 1
    dh = d // c.n_heads
    lin = c.attention == "linear"
    tile = 0 if d >= 512 else 64          # module kernel: groups of up to 64 rows, d <= 256
    rows_item = sum(U)
    out = {k: 0.0 for k in fam_names}

    def add(fam, v):
        out[fam] = out.get(fam, 0.0) + v

    fused = "layer" in fam_names or "post" in fam_names

    def selfattn(group):   # q|k|v projection inside the attention kernel (d = 128, head width 32)
        return fused and d == 128 and d // c.n_heads == 32 and group <= 256

    def lin_state(keys):   # state of every head over `keys` key rows (z included)
        return 2.0 * keys * d * dh + keys * d

    def lin_apply(queries):
        return 2.0 * queries * d * (dh + 1)

    for name, (rows, groups, size, first) in (("ctx", (B * T, B, T, False)), ("seq", (B * K * S, B * K, S, True)),
                                              ("cross", (B * K, B, K, False))):
        proj, attn, tail = module_parts(d, F, n, rows, groups, size, first)
        if lin and name != "seq":
            add("gemm", proj)
            add("linear", n * (lin_state(rows) + lin_apply(rows)))
            add("post" if fused else "gemm", tail)
        elif fused and size <= tile:
            add("layer", proj + attn + tail)
        elif fused:
            add("attention" if selfattn(size) else "gemm", proj)
            add("attention", attn)
            add("post", tail)
        else:
            add("gemm", proj + tail)
            add("attention", attn)
    # key/value cache of the item layers: in the last context tail when that tail is fused
    add("post" if fused and (lin or T > tile) else "gemm", 4.0 * n * B * T * d * d)
    if lin:
        add("linear", n * lin_state(B * T))       # the cache's per-head state, per item layer
    # distinct items: q|k|v, self-attention, output + query projections, cross-attention, FFN
    add("attention", sum(n * 4.0 * u * u * d for u in U))
    if lin:
        add("linear", n * lin_apply(rows_item))
    else:
        add("attention", sum(n * 4.0 * u * T * d for u in U))
    ucap = min(c.M, K * c.L)
    add("attention" if selfattn(ucap) else "gemm", n * 6.0 * d * d * rows_item)
    # output + query projections of the item self-attention: inside the fused cross-attention
    # kernel when it applies (softmax, groups and context of at most 256 rows), else in the tail
    cross_fused = selfattn(ucap) and not lin and T <= 256
    add("attention" if cross_fused else ("post" if fused else "gemm"), n * 4.0 * d * d * rows_item)
    add("post" if fused else "gemm", n * (2.0 * d * d + 4.0 * d * F) * rows_item)
    return out


def linear_bytes(c, U):
    """Algorithmic HBM bytes of the linear-attention kernels in one pass: each state kernel reads
    the keys and values once and writes the fp32 state; each apply kernel reads the queries and
    the state and writes the output rows."""
    d, n, B, T, K = c.d, c.n_layers, c.B, c.T, c.K
    H, dh = c.n_heads, c.d // c.n_heads
    esz = 2 if c.dtype == "bf16" else 4
    st = lambda groups: groups * H * (dh + 1) * dh * 4
    total = 0.0
    for rows, groups in ((B * T, B), (B * K, B)):                 # context, cross-sequence modules
        total += n * (2 * rows * d * esz + st(groups) + rows * d * esz + st(groups) + rows * d * esz)
    total += n * (2 * B * T * d * esz + st(B))                     # the item layers' context state
    total += n * (2 * sum(U) * d * esz + st(B))                    # the items' cross-attention
    return total


def naive_flops(c, U):
    """Algorithmic flops of the candidate-factorised evaluator (context encoded once per list,
    distinct-element set encoded once per element occurrence; SeqEnc, cross-sequence module as
    in the joint pass)."""
    d, F, n, B, T, K, L, S = c.d, c.ffn, c.n_layers, c.B, c.T, c.K, c.L, c.L + 1
    ctx = sum(module_parts(d, F, n, T, 1, T)) + 4.0 * n * T * d * d
    items = [n * (4.0 * u * u * d + 4.0 * u * T * d) + n * (12.0 * d * d + 4.0 * d * F) * u for u in U]
    seq = sum(module_parts(d, F, n, B * K * S, B * K, S, True))
    cross = sum(module_parts(d, F, n, B * K, B, K))
    return B * K * ctx + K * L * sum(items) + seq + cross


def train_flops(c, U):
    """Algorithmic flops of one training step (forward + backward) over the valid rows: every
    product of the forward once, and twice more in the backward (input and weight gradients of a
    projection; dP, dV, dQ, dK of an attention).  U: distinct elements per request."""
    d, F, H, n, dh = c.d, c.ffn, c.n_heads, c.n_layers, c.d // c.n_heads
    B, T, K, S = c.B, c.T, c.K, c.L + 1
    Usum = float(sum(U))

    def enc(rows, att):                      # one encoder block: projections, FFN, attention
        return 2 * rows * (4 * d * d + 2 * d * F) + att
    fwd = n * enc(B * T, 4 * B * H * T * T * dh)
    fwd += n * 2 * (2 * B * T * d * d)                                  # context keys and values per item layer
    fwd += n * (2 * Usum * (6 * d * d + 2 * d * F)
                + 4 * H * dh * sum(u * u + u * T for u in U))          # item-set layers
    fwd += n * enc(B * K * S, 4 * B * K * H * S * S * dh)              # SeqEnc
    fwd += n * enc(B * K, 4 * B * H * K * K * dh)                      # cross-sequence module
    fwd += 2 * B * K * d
    return 3 * fwd


def cpu_baseline(c, W, I, seconds: float):
    """The float64 oracle, in its candidate-factorised order, on this host for a bounded time.

    Whole lists are evaluated one after another, request by request in batch order (for each
    list the context is re-encoded, the item set re-encoded for each of its L occurrences, then
    SeqEnc), until `seconds` have passed; lists/s is the count over the elapsed time.  The
    cross-sequence module and head, which the oracle runs once per request over all K lists,
    are not part of the sample.
    """
    import numpy as np
    import oracle
    ev = oracle.evaluator
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"] or [1])
    except Exception:
        threads = len(os.sched_getaffinity(0))
    done, reqs, t0 = 0, 0, time.perf_counter()
    for b in range(c.B):
        if time.perf_counter() - t0 >= seconds:
            break
        req = {k: (None if v is None else v[b:b + 1]) for k, v in I.items()}
        lists_b = np.asarray(req["lists"][0])
        reqs += 1
        for k in range(c.K):
            if time.perf_counter() - t0 >= seconds:
                break
            _, kv = ev.encode_context(c, W, ev.context_rows(c, W, req, 0))
            rows = np.empty((c.L, c.d))
            for j in range(c.L):
                uniq, _ = ev.distinct_items(lists_b)
                H = ev.encode_items(c, W, ev.item_rows(c, W, req, 0, uniq), kv)
                rows[j] = H[int(np.searchsorted(uniq, lists_b[k, j]))]
            ev.encode_sequence(c, W, ev.assemble_one(W, rows))
            done += 1
    dt = time.perf_counter() - t0
    cpu = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": round(done / dt, 3), "unit": "lists/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{done} lists of the first {reqs} request(s) (float64 numpy, candidate-factorised order: context "
                      f"re-encoded per list, item set re-encoded per occurrence) in {dt:.1f} s on {cpu}"}


def cpu_cached(c, W, I, seconds: float):
    """The same float64 oracle in the joint order (context and item set encoded once per request,
    then every list): the evaluator the paper deploys, on this host's cores.  Whole requests are
    evaluated in batch order until `seconds` have passed (at least one); lists/s = K * requests /
    elapsed time."""
    import oracle
    done, t0 = 0, time.perf_counter()
    for b in range(c.B):
        if done and time.perf_counter() - t0 >= seconds:
            break
        oracle.evaluate_cached(c, W, I, requests=[b])
        done += 1
    dt = time.perf_counter() - t0
    return {"value": round(c.K * done / dt, 3), "unit": "lists/s", "kind": "oracle, joint order",
            "sample": f"{done} request(s) x {c.K} lists (float64 numpy, context and item set encoded once per "
                      f"request) in {dt:.1f} s"}


# Sources that define each profiled family's kernels (and api.cpp, which sets their arguments):
# a traffic profile is used only while all of them are unchanged.
TRAFFIC_SOURCES = {
    "layer": ("layer.hip", "fe_tile.h", "fe_common.h", "api.cpp"),
    "seq_module": ("layer.hip", "fe_tile.h", "fe_common.h", "api.cpp"),
    "post": ("layer.hip", "fe_tile.h", "fe_common.h", "api.cpp"),
    "attention": ("attn_fused.hip", "attention.hip", "fe_dedup.h", "fe_tile.h", "fe_common.h", "api.cpp"),
}
# kernel-name prefixes of each family (as rocprofv3 reports them)
TRAFFIC_KERNELS = {
    "layer": ("k_module_small",),
    "seq_module": ("k_module_small",),        # its [CLS]-only instantiations (template flag `true`)
    "post": ("k_post",),
    "attention": ("k_self_attention", "k_cross_attention", "k_attention"),
}


def traffic_kernel(family: str, name: str) -> bool:
    """Whether rocprofv3 kernel `name` belongs to `family`."""
    n = name.replace("void (anonymous namespace)::", "")
    if not any(n.startswith(p) for p in TRAFFIC_KERNELS[family]):
        return False
    return family != "seq_module" or ", true," in n


def sources_digest(family: str) -> str:
    """sha256 over the sources of `family`'s kernels (identifies the kernels a traffic profile saw)."""
    import hashlib
    h = hashlib.sha256()
    for f in TRAFFIC_SOURCES[family]:
        with open(os.path.join(ROOT, "paper_2603_02565_amd", "csrc", f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()


def measured_traffic(family: str):
    """HBM bytes per launch of `family` from profiles/traffic.json, if it was taken on these sources.

    The file holds FETCH_SIZE and WRITE_SIZE (rocprofv3 --pmc, one pass each) per dispatch of the
    family's kernels, each scaled by the factor the same counter shows for a plain copy of known
    size; a family's entry is ignored (null) once its kernels' sources have changed.
    """
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    entry = t.get("families", {}).get(family)
    if family not in TRAFFIC_SOURCES or not entry or entry.get("sources_sha256") != sources_digest(family):
        return None
    return entry.get("bytes_per_launch")


MATRIX_FAMILIES = ("gemm", "ffn", "attention", "layer", "post")


def stage_table(c, U, fam, steps):
    """Per kernel family: time per step, launches, mean launch time; TFLOP/s and the MFMA
    fraction of the matrix-product families; GB/s and the HBM fraction of the linear-attention
    kernels (bandwidth-bound: a few flops per byte of keys, values and queries)."""
    stages = {}
    for name, (ms, n) in fam.items():
        if n == 0:
            continue
        stages[name] = {"ms_per_step": round(ms / steps, 5), "launches_per_step": n // steps,
                        "avg_launch_us": round(ms * 1e3 / n, 3)}
    peak = PEAK_BF16_TFLOPS if c.dtype == "bf16" else PEAK_FP32_TFLOPS
    flops = family_flops(c, U, set(stages))
    for name in MATRIX_FAMILIES:
        if name in stages and flops.get(name, 0.0) > 0:
            tf = flops[name] / (fam[name][0] / steps / 1e3) / 1e12
            stages[name].update(tflops=round(tf, 2), mfma_frac=round(tf / peak, 4))
    if "linear" in stages:
        nbytes = linear_bytes(c, U)
        gbs = nbytes / (fam["linear"][0] / steps / 1e3) / 1e9
        stages["linear"].update(bytes_per_step=int(nbytes), GBps=round(gbs, 1), hbm_frac=round(gbs / PEAK_HBM_GBS, 4),
                                gflops_per_step=round(flops.get("linear", 0.0) / 1e9, 3))
    return stages, flops


def time_pass(step, stream, steps, warmup):
    """Mean device time of `steps` back-to-back passes (after `warmup`), in ms."""
    import torch
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def graph_us(fn, stream, reps: int = ASM_REPS, replays: int = 5) -> float:
    """Mean duration of one call of `fn` when `reps` calls run back to back on the device: the calls
    are captured as one HIP graph and the graph is replayed `replays` times between two events (no
    per-launch event or host call in between), in microseconds."""
    import torch
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(reps):
            fn()
    g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(replays):
        g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / (replays * reps)
    del g
    return us


def assemble_entry(c, U, ev, bufs, stream):
    """The assembly alone (fe_assemble back to back from a HIP graph) against its algorithmic bytes,
    beside two reference points timed the same way: torch's fill of a tensor the size of seq (the
    write-only floor: the assembly writes those bytes and reads less than a tenth as much) and
    torch's copy of it (read + write)."""
    import torch
    from paper_2603_02565_amd import flasheval as fe
    b = bufs
    asm_us = graph_us(lambda: fe.fe_assemble(ev.handle, c.B, c.K, c.L, b["U_cap"], b["slot"], b["H"], b["seq"]), stream)
    nbytes = assemble_bytes(c, U)
    scratch = torch.empty_like(b["seq"])
    seq_bytes = scratch.numel() * scratch.element_size()
    fill_us = graph_us(lambda: scratch.fill_(0.5), stream)
    copy_us = graph_us(lambda: scratch.copy_(b["seq"]), stream)
    del scratch
    gbs = nbytes / (asm_us / 1e6) / 1e9
    return {"avg_launch_us": round(asm_us, 3), "bytes_per_launch": int(nbytes), "GBps": round(gbs, 1),
            "hbm_frac": round(gbs / PEAK_HBM_GBS, 4),
            "timing": f"mean of {5 * ASM_REPS} back-to-back launches replayed from a HIP graph",
            "write_floor": {"avg_launch_us": round(fill_us, 3), "bytes_per_launch": seq_bytes,
                            "GBps": round(seq_bytes / (fill_us / 1e6) / 1e9, 1),
                            "what": "torch fill_ of a tensor the size of seq (write only), timed the same way"},
            "copy_reference": {"avg_launch_us": round(copy_us, 3), "bytes_per_launch": 2 * seq_bytes,
                               "GBps": round(2 * seq_bytes / (copy_us / 1e6) / 1e9, 1),
                               "what": "torch copy_ of a tensor the size of seq (read + write), timed the same way"}}


def workload_entry(c, steps: int, warmup: int, trace: bool = True, cpu_seconds: float = 0.0):
    """One workload's pass on this GPU: time per batch (events over `steps` back-to-back passes) and
    its median over per-pass events, lists/s, the measured distinct-element counts, the item stage
    (fe_encode_items) timed alone, the assembly against its write-only floor, the dominant
    matrix-product kernel family with its TFLOP/s (per-launch trace times scaled to the untraced
    pass), and with `cpu_seconds` > 0 the oracle timed on the same workload."""
    import numpy as np
    import torch
    import gen
    from paper_2603_02565_amd import flasheval as fe
    W, I = gen.make_weights(c), gen.make_inputs(c)
    ev = fe.Evaluator(c.d, c.n_heads, c.n_layers, c.ffn, c.max_L, c.vocab, c.dtype, W, attention=c.attention)
    bufs = ev.allocate(c.B, c.T, c.M, c.K, c.L)
    act = torch.bfloat16 if c.dtype == "bf16" else torch.float32
    dev = torch.device("cuda", 0)
    x = None if I["x"] is None else torch.from_numpy(I["x"]).to(dev).to(act)
    pool = None if I["pool"] is None else torch.from_numpy(I["pool"]).to(dev).to(act)
    ids = None if I["ctx_ids"] is None else torch.from_numpy(I["ctx_ids"]).to(dev)
    lists = torch.from_numpy(I["lists"]).to(dev)
    stream = torch.cuda.current_stream()
    b = bufs

    def step():
        ev.run(x=x, ctx_ids=ids, pool=pool, lists=lists)

    ms = time_pass(step, stream, steps, warmup)
    sets = [b] + [ev.allocate(c.B, c.T, c.M, c.K, c.L) for _ in range(PIPE_STREAMS - 1)]
    ex = fe.Executor(ev, PIPE_STREAMS)
    n_sub = [0]

    def submit():
        ex.submit(sets[n_sub[0] % PIPE_STREAMS], x=x, ctx_ids=ids, pool=pool, lists=lists)
        n_sub[0] += 1

    for _ in range(max(warmup, PIPE_STREAMS)):
        submit()
    ex.join()
    torch.cuda.synchronize()
    q0, q1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    q0.record(stream)
    for _ in range(steps):
        submit()
    ex.join()
    q1.record(stream)
    torch.cuda.synchronize()
    pipe_ms = q0.elapsed_time(q1) / steps
    ex.close()
    del sets
    ev.buffers = b
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    evs[0].record(stream)
    for i in range(steps):
        step()
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    p50 = float(np.median([evs[i].elapsed_time(evs[i + 1]) for i in range(steps)]))
    U = b["n_uniq"].cpu().numpy().tolist()
    items_us = time_pass(lambda: fe.fe_encode_items(ev.handle, c.B, c.M, pool, lists, c.K, c.L, b["kv"], c.T, b["uniq"],
                                                    b["n_uniq"], b["slot"], b["H"], b["ws"]),
                         stream, steps, warmup) * 1e3
    entry = {"workload": c.label, "B": c.B, "T": c.T, "d": c.d, "K": c.K, "L": c.L, "M": c.M,
             "attention": c.attention, "lists_per_batch": c.B * c.K, "ms_per_batch": round(ms, 5),
             "lists_per_s": round(c.B * c.K / (ms / 1e3), 1), "p50_ms": round(p50, 5),
             "pipelined": {"streams": PIPE_STREAMS, "ms_per_batch": round(pipe_ms, 5),
                           "lists_per_s": round(c.B * c.K / (pipe_ms / 1e3), 1)},
             "U_mean": round(float(np.mean(U)), 2),
             "rho": round(c.K * c.L / float(np.mean(U)), 3), "item_stage_us": round(items_us, 2),
             "assemble": assemble_entry(c, U, ev, b, stream)}
    if trace:
        fe.fe_trace_enable(True)
        for _ in range(steps):
            step()
        torch.cuda.synchronize()
        fam = fe.fe_trace_read()
        fe.fe_trace_enable(False)
        fam = {k: v for k, v in fam.items() if v[1] > 0}
        traced = sum(v[0] for v in fam.values()) / steps
        scale = min(1.0, ms / traced) if traced > 0 else 1.0
        flops = family_flops(c, U, set(fam))
        peak = PEAK_BF16_TFLOPS if c.dtype == "bf16" else PEAK_FP32_TFLOPS
        mm = {k: v for k, v in fam.items() if k in MATRIX_FAMILIES and flops.get(k, 0.0) > 0}
        if mm:
            dom = max(mm, key=lambda k: mm[k][0])
            t_ms = mm[dom][0] / steps * scale
            tf = flops[dom] / (t_ms / 1e3) / 1e12
            entry["dominant_family"] = {"family": dom, "ms_per_batch": round(t_ms, 5), "tflops": round(tf, 2),
                                        "mfma_frac": round(tf / peak, 4), "share_of_pass": round(t_ms / ms, 4)}
            mm_ms = sum(v[0] for v in mm.values()) / steps * scale
            entry["mfma_util_matrix_stages"] = round(sum(flops[k] for k in mm) / (mm_ms / 1e3) / 1e12 / peak, 4)
    if cpu_seconds > 0:
        entry["cpu_baseline"] = cpu_baseline(c, W, I, cpu_seconds)
    ev.close()
    del bufs, x, pool, ids, lists
    torch.cuda.empty_cache()
    return entry


def copy_calibration() -> int:
    """A plain elementwise copy of 256 MiB (fp32 x 1.0), three times: reads and writes 256 MiB each."""
    import torch
    n = 64 << 20
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        torch.mul(src, 1.0, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": n * 4}), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", type=int, default=1, choices=[1, 2, 3, 4])
    ap.add_argument("--K", type=int, default=None, help="lists per request for workload 2")
    ap.add_argument("--attention", choices=["softmax", "linear"], default="softmax",
                    help="attention form of the model (linear: the kernelized variant of Appendix B.3)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-trace", action="store_true", help="skip the traced pass (for profiler runs)")
    ap.add_argument("--no-graph", action="store_true", help="skip the graph-replay timing (for profiler runs)")
    ap.add_argument("--no-naive", action="store_true",
                    help="skip timing the candidate-factorised evaluator (no reuse) on the GPU")
    ap.add_argument("--naive-steps", type=int, default=5)
    ap.add_argument("--no-train", action="store_true", help="skip the fp32 training-step timing")
    ap.add_argument("--train-steps", type=int, default=10)
    ap.add_argument("--no-variants", action="store_true",
                    help="skip timing the pass without cross-sequence interaction (for profiler runs)")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the K sweep and the long-context / text-hypothesis workloads after the headline run")
    ap.add_argument("--no-pipeline", action="store_true",
                    help="skip the pipelined-executor throughput (for profiler runs of single kernels)")
    ap.add_argument("--cpu-all", action="store_true",
                    help="also time the oracle (candidate-factorised order, --cpu-seconds each) on every K-sweep "
                         "and long-context / text-hypothesis workload")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 256 MiB copy (to scale rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    args = ap.parse_args()
    if args.copy_calibration:
        return copy_calibration()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (the joint pass shards over independent requests; "
              f"see DESIGN.md); got --gpus {args.gpus}", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import gen
    from paper_2603_02565_amd import flasheval as fe

    if not torch.cuda.is_available():
        print("bench.py needs an MI355X", file=sys.stderr)
        return 1
    torch.cuda.set_device(0)
    c = gen.config(args.workload, K=args.K) if args.workload == 2 else gen.config(args.workload)
    c = replace(c, attention=args.attention)
    W, I = gen.make_weights(c), gen.make_inputs(c)
    ev = fe.Evaluator(c.d, c.n_heads, c.n_layers, c.ffn, c.max_L, c.vocab, c.dtype, W, attention=c.attention)
    bufs = ev.allocate(c.B, c.T, c.M, c.K, c.L)
    act = torch.bfloat16 if c.dtype == "bf16" else torch.float32
    dev = torch.device("cuda", 0)
    x = None if I["x"] is None else torch.from_numpy(I["x"]).to(dev).to(act)
    pool = None if I["pool"] is None else torch.from_numpy(I["pool"]).to(dev).to(act)
    ids = None if I["ctx_ids"] is None else torch.from_numpy(I["ctx_ids"]).to(dev)
    lists = torch.from_numpy(I["lists"]).to(dev)
    stream = torch.cuda.current_stream()

    def step():
        ev.run(x=x, ctx_ids=ids, pool=pool, lists=lists)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # ---- timed region: K whole passes back to back on one stream, an event between consecutive
    # passes (the metric: B*K lists over the device time of the five calls for one batch)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    evs[0].record(stream)
    for i in range(args.steps):
        step()
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per_step = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)])
    ms_per_step = evs[0].elapsed_time(evs[-1]) / args.steps
    lists_per_s = c.B * c.K / (ms_per_step / 1e3)

    # ---- serving throughput beside it: K passes (each over the whole batch) submitted round-robin
    # to the pipelined executor, PIPE_STREAMS batches in flight, one buffer set per stream
    pipe_ms = None
    if not args.no_pipeline:
        pipe_sets = [bufs] + [ev.allocate(c.B, c.T, c.M, c.K, c.L) for _ in range(PIPE_STREAMS - 1)]
        ex = fe.Executor(ev, PIPE_STREAMS)

        def submit(i):
            ex.submit(pipe_sets[i % PIPE_STREAMS], x=x, ctx_ids=ids, pool=pool, lists=lists)

        for i in range(max(args.warmup, PIPE_STREAMS)):
            submit(i)
        ex.join()
        torch.cuda.synchronize()
        p0, p1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        p0.record(stream)
        for i in range(args.steps):
            submit(i)
        ex.join()
        p1.record(stream)
        torch.cuda.synchronize()
        pipe_ms = p0.elapsed_time(p1) / args.steps
        ex.close()
        del pipe_sets
        ev.buffers = bufs
        step()                 # leave this stream's pass outputs in the buffers
        torch.cuda.synchronize()

    U = bufs["n_uniq"].cpu().numpy().tolist()
    asm_bytes = assemble_bytes(c, U)

    # ---- the pass without cross-sequence interaction (SeqEnc output scored directly)
    no_cross_ms = None
    C_ind = torch.empty((c.B, c.K, c.d), dtype=torch.float32, device=dev)

    def step_no_cross():
        b, h = bufs, ev.handle
        fe.fe_encode_context(h, c.B, c.T, x, ids, b["kv"], b["ws"])
        fe.fe_encode_items(h, c.B, c.M, pool, lists, c.K, c.L, b["kv"], c.T, b["uniq"], b["n_uniq"], b["slot"], b["H"],
                           b["ws"])
        fe.fe_assemble(h, c.B, c.K, c.L, b["U_cap"], b["slot"], b["H"], b["seq"])
        fe.fe_encode_sequences(h, c.B, c.K, c.L, b["seq"], C_ind, b["ws"])
        fe.fe_score_select(h, c.B, c.K, C_ind, b["scores"], b["best"])

    if not args.no_variants:
        for _ in range(args.warmup):
            step_no_cross()
        v0, v1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        v0.record(stream)
        for _ in range(args.steps):
            step_no_cross()
        v1.record(stream)
        torch.cuda.synchronize()
        no_cross_ms = v0.elapsed_time(v1) / args.steps
        step()                 # leave the full pass's outputs in the buffers
        torch.cuda.synchronize()

    # ---- the same pass captured once as a HIP graph and replayed K times
    graph_ms = None
    if not args.no_graph:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        for _ in range(args.warmup):
            graph.replay()
        torch.cuda.synchronize()
        g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        g0.record(stream)
        for _ in range(args.steps):
            graph.replay()
        g1.record(stream)
        torch.cuda.synchronize()
        graph_ms = g0.elapsed_time(g1) / args.steps
        del graph

    # ---- the assembly alone, against its write-only floor and a copy of the same size
    asm_entry = assemble_entry(c, U, ev, bufs, stream) if not args.no_trace else None

    # ---- kernel-timing region: the same steps with HIP events around every launch
    fam = {}
    launches = []
    if not args.no_trace:
        fe.fe_trace_enable(True)
        for _ in range(args.steps):
            step()
        torch.cuda.synchronize()
        launches = fe.fe_trace_read_launches()
        fe.fe_trace_enable(False)
        for f, t in launches:
            ms_n = fam.get(f, (0.0, 0))
            fam[f] = (ms_n[0] + t, ms_n[1] + 1)
    # the pass's launch sequence (identical every step) and the mean time of each of its launches
    per_pass = len(launches) // args.steps if launches else 0
    seq_fams = [f for f, _ in launches[:per_pass]]
    pos_ms = [float(np.mean([launches[i * per_pass + j][1] for i in range(args.steps)])) for j in range(per_pass)] \
        if per_pass and len(launches) == per_pass * args.steps and \
        all([f for f, _ in launches[i * per_pass:(i + 1) * per_pass]] == seq_fams for i in range(args.steps)) else []
    # the SeqEnc module: the one "layer" launch right after the assembly (whole sequence encoder in
    # one kernel); timed on its own as back-to-back fe_encode_sequences calls between two events
    seq_pos = None
    if pos_ms and "assemble" in seq_fams:
        a = len(seq_fams) - 1 - seq_fams[::-1].index("assemble")
        if a + 1 < len(seq_fams) and seq_fams[a + 1] == "layer":
            seq_pos = a + 1
    seqenc_us = None
    if seq_pos is not None:
        C_out = torch.empty((c.B, c.K, c.d), dtype=torch.float32, device="cuda")

        def seq_only():
            fe.fe_encode_sequences(ev.handle, c.B, c.K, c.L, bufs["seq"], C_out, bufs["ws"])

        seqenc_us = time_pass(seq_only, stream, max(50, args.steps), 5) * 1e3
        del C_out

    out = {
        "metric": METRIC, "value": round(lists_per_s, 1), "unit": "lists/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": c.dtype,
        "data": "synthetic (seeded; random-init weights)",
        "config": {"workload": f"{c.name}: B={c.B} T={c.T} d={c.d} heads={c.n_heads} layers={c.n_layers} "
                               f"F={c.ffn} M={c.M} K={c.K} L={c.L}"
                               + (" (linear attention)" if c.attention == "linear" else ""),
                   "B": c.B, "T": c.T, "d": c.d, "M": c.M, "K": c.K, "L": c.L, "parallelism": "none (1 GPU)"},
        "p50_ms": round(float(np.percentile(per_step, 50)), 5),
        "p90_ms": round(float(np.percentile(per_step, 90)), 5),
        "wall_ms_per_step": round(wall * 1e3 / args.steps, 5),
        "pipelined": None if pipe_ms is None else {
            "streams": PIPE_STREAMS, "ms_per_step": round(pipe_ms, 5), "value": round(c.B * c.K / (pipe_ms / 1e3), 1),
            "what": "serving throughput: K passes (each over the whole batch) submitted round-robin to the library's "
                    "pipelined executor (fe_executor_*), one buffer set per stream, timed between two events around "
                    "all K; value above is one batch at a time on one stream"},
        "without_cross_sequence": None if no_cross_ms is None else {
            "ms_per_step": round(no_cross_ms, 5), "value": round(c.B * c.K / (no_cross_ms / 1e3), 1)},
        "graph_replay": None if graph_ms is None else {"ms_per_step": round(graph_ms, 5),
                                                       "value": round(c.B * c.K / (graph_ms / 1e3), 1)},
        "U_mean": round(float(np.mean(U)), 2), "rho": round(c.K * c.L / float(np.mean(U)), 3),
    }
    if fam:
        peak = PEAK_BF16_TFLOPS if c.dtype == "bf16" else PEAK_FP32_TFLOPS
        stages, flops = stage_table(c, U, fam, args.steps)
        if "assemble" in stages and asm_entry is not None:
            # per-launch events add their own overhead to a kernel this short: the back-to-back
            # average from the graph of assembly launches is the duration the fraction uses
            traced_us = stages["assemble"]["avg_launch_us"]
            stages["assemble"].update(asm_entry)
            stages["assemble"]["traced_avg_launch_us"] = traced_us
        dom = max((k for k in stages if k != "linear"), key=lambda k: stages[k]["ms_per_step"])
        dom_ms, dom_n = fam[dom]
        avg_s = dom_ms / dom_n / 1e3
        longest = int(np.argmax(pos_ms)) if pos_ms else None
        if longest is not None and longest == seq_pos and seqenc_us is not None:
            # the dominant kernel is the SeqEnc module: its own flops over its own back-to-back time
            S = c.L + 1
            sf = sum(module_parts(c.d, c.ffn, c.n_layers, c.B * c.K * S, c.B * c.K, S, True))
            ach = sf / (seqenc_us / 1e6) / 1e12
            out["roofline"] = {"kernel": "k_module_small (SeqEnc module)", "bound": "mfma", "achieved": round(ach, 2),
                               "peak": round(peak, 1), "unit": "TFLOP/s", "frac": round(ach / peak, 4),
                               "traffic": measured_traffic("seq_module"), "avg_launch_us": round(seqenc_us, 3),
                               "launches_per_step": 1, "flops_per_launch": int(sf),
                               "share_of_pass": round(pos_ms[longest] / sum(pos_ms), 4),
                               "timing": "mean of back-to-back fe_encode_sequences calls (one launch each) "
                                         "between two HIP events on the pass's stream"}
        elif flops.get(dom, 0.0) > 0:
            per_launch = flops[dom] / (dom_n / args.steps)
            ach = per_launch / avg_s / 1e12
            out["roofline"] = {"kernel": dom, "bound": "mfma", "achieved": round(ach, 2), "peak": round(peak, 1),
                               "unit": "TFLOP/s", "frac": round(ach / peak, 4), "traffic": measured_traffic(dom),
                               "avg_launch_us": round(avg_s * 1e6, 3), "launches_per_step": dom_n // args.steps}
        else:
            per_launch = asm_bytes
            ach = per_launch / avg_s / 1e9
            out["roofline"] = {"kernel": dom, "bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS,
                               "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4), "traffic": measured_traffic(dom),
                               "avg_launch_us": round(avg_s * 1e6, 3), "launches_per_step": dom_n // args.steps}
        mm_fams = [k for k in MATRIX_FAMILIES if k in stages]
        traced_ms = sum(v[0] for v in fam.values()) / args.steps
        # each per-launch event pair adds its own overhead (about 2 us), so the traced kernel times
        # sum to more than the untraced pass; the matrix stages' time is taken as their traced share
        # of the untraced pass time (the pass runs its kernels back to back)
        scale = min(1.0, ms_per_step / traced_ms) if traced_ms > 0 else 1.0
        mm_ms = sum(fam[k][0] for k in mm_fams) / args.steps * scale
        mm_flops = sum(flops.get(k, 0.0) for k in mm_fams)
        out["mfma_util_matrix_stages"] = round(mm_flops / (mm_ms / 1e3) / 1e12 / peak, 4)
        out["mfma_util_timing"] = (f"matrix-stage kernel time = their share of the traced kernel time x the untraced "
                                   f"pass time (scale {scale:.3f}); flops algorithmic")
        for k in mm_fams:
            if "tflops" in stages[k]:
                tf = stages[k]["tflops"] / scale
                stages[k].update(tflops_event_corrected=round(tf, 2), mfma_frac_event_corrected=round(tf / peak, 4))
        out["kernel_ms_per_step"] = round(traced_ms, 5)
        out["stages"] = stages
    if not args.no_variants and c.attention == "softmax":
        # the linear-attention variant (the deployment setting of Appendix B.3) on the same weights
        # and inputs: same shapes, the context, item->context and cross-sequence attention linear
        cl = replace(c, attention="linear")
        ev_lin = fe.Evaluator(c.d, c.n_heads, c.n_layers, c.ffn, c.max_L, c.vocab, c.dtype, W, attention="linear")
        ev_lin.allocate(c.B, c.T, c.M, c.K, c.L)

        def step_lin():
            ev_lin.run(x=x, ctx_ids=ids, pool=pool, lists=lists)

        lin_ms = time_pass(step_lin, stream, args.steps, args.warmup)
        entry = {"ms_per_step": round(lin_ms, 5), "value": round(c.B * c.K / (lin_ms / 1e3), 1),
                 "what": "same workload with linear attention (phi = elu + 1) in the context, item->context and "
                         "cross-sequence attention; the context cache is the per-head state"}
        if not args.no_trace:
            fe.fe_trace_enable(True)
            for _ in range(args.steps):
                step_lin()
            torch.cuda.synchronize()
            lfam = fe.fe_trace_read()
            fe.fe_trace_enable(False)
            entry["stages"], _ = stage_table(cl, U, lfam, args.steps)
        out["linear_attention"] = entry
        ev_lin.close()
        torch.cuda.empty_cache()
    if not args.no_naive:
        # the same network with every reuse taken out (fe_evaluate_naive), same inputs, same GPU
        ev.allocate_naive(c.B, c.T, c.M, c.K, c.L, token_ids=ids is not None)

        def naive_step():
            ev.run_naive(x=x, ctx_ids=ids, pool=pool, lists=lists)

        naive_step()
        torch.cuda.synchronize()
        n0, n1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        n0.record(stream)
        for _ in range(args.naive_steps):
            naive_step()
        n1.record(stream)
        torch.cuda.synchronize()
        naive_ms = n0.elapsed_time(n1) / args.naive_steps
        same = bool(torch.equal(ev.naive_buffers["best"], bufs["best"]))
        jf = sum(family_flops(c, U, {"layer", "post", "attention", "gemm"}).values())
        nf = naive_flops(c, U)
        out["naive_gpu"] = {
            "ms_per_step": round(naive_ms, 4), "value": round(c.B * c.K / (naive_ms / 1e3), 1), "unit": "lists/s",
            "steps": args.naive_steps, "t_joint_over_t_ind": round(ms_per_step / naive_ms, 6),
            "flops_joint_over_ind": round(jf / nf, 6), "one_over_rho": round(float(np.mean(U)) / (c.K * c.L), 4),
            "tflops": round(nf / (naive_ms / 1e3) / 1e12, 1), "same_selection": same,
            "what": "context encoded once per list, distinct-element set once per element occurrence, "
                    "each list assembled from its own encodings (fe_evaluate_naive)"}
        ev.naive_buffers = None
        torch.cuda.empty_cache()
    if not args.no_train and c.attention == "softmax" and c.K <= 1024:
        # one training step (Section 4.5) on the same batch: fp32 model, listwise CE loss
        cfg = fe.fe_config(c.d, c.n_heads, c.n_layers, c.ffn, c.max_L, c.vocab, fe.FE_F32, fe.FE_ATTN_SOFTMAX)
        Pt = torch.from_numpy(fe.pack_params(W, c.n_layers, c.vocab)).to(dev)
        Gt = torch.empty_like(Pt)
        xt = None if I["x"] is None else torch.from_numpy(I["x"]).to(dev).float()
        pt = None if I["pool"] is None else torch.from_numpy(I["pool"]).to(dev).float()
        rel = torch.from_numpy(gen.make_relevance(c)).to(dev)
        loss_t = torch.empty(1, device=dev)
        wst = torch.empty(fe.fe_train_workspace_size(cfg, c.B, c.T, c.M, c.K, c.L), dtype=torch.uint8, device=dev)

        def train_step():
            fe.fe_train_grads(cfg, Pt, c.B, c.T, c.M, c.K, c.L, xt, ids, pt, lists, rel, fe.FE_LOSS_CE, loss_t, None,
                              Gt, wst)

        tr_ms = time_pass(train_step, stream, args.train_steps, 2)
        tf = train_flops(c, U)
        out["train"] = {
            "ms_per_step": round(tr_ms, 3), "steps_per_s": round(1e3 / tr_ms, 2),
            "lists_per_s": round(c.B * c.K / (tr_ms / 1e3), 1), "loss": round(float(loss_t.item()), 6),
            "dtype": "f32", "loss_kind": "ce", "steps": args.train_steps,
            "gflops_per_step": round(tf / 1e9, 2), "tflops": round(tf / (tr_ms / 1e3) / 1e12, 2),
            "frac_of_fp32_peak": round(tf / (tr_ms / 1e3) / 1e12 / PEAK_FP32_TFLOPS, 4),
            "workspace_GiB": round(wst.numel() / 2**30, 3),
            "what": "fe_train_grads: forward with saved activations, listwise CE loss, backward of every "
                    "parameter, on this batch in fp32"}
        del Pt, Gt, wst
        torch.cuda.empty_cache()
    if not args.no_sweep and args.workload == 1:
        # the other workloads on the same GPU in the same run: the K sweep on the RecSys-base shapes
        # (Section 5.2: the item stage follows the distinct elements, not the K*L occurrences), the
        # long-context workload (softmax and linear attention) and the text-hypothesis workload
        n_steps = max(10, min(args.steps, 30))
        ev.close()
        del bufs
        torch.cuda.empty_cache()
        cs = args.cpu_seconds if args.cpu_all else 0.0
        out["k_sweep"] = [workload_entry(gen.config(2, K=k), n_steps, 5, trace=not args.no_trace, cpu_seconds=cs)
                          for k in gen.K_SWEEP]
        out["workloads"] = [workload_entry(gen.config(3), n_steps, 5, trace=not args.no_trace, cpu_seconds=cs),
                            workload_entry(gen.config(3, attention="linear"), n_steps, 5, trace=not args.no_trace),
                            workload_entry(gen.config(4), n_steps, 5, trace=not args.no_trace, cpu_seconds=cs)]
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(c, W, I, args.cpu_seconds)
        out["cpu_baseline"]["joint_order"] = cpu_cached(c, W, I, args.cpu_seconds / 3)
    ev.close()
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
