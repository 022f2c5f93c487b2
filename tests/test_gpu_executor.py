"""The pipelined executor (fe_executor_*): whole passes of independent batches round-robin over
the library's own streams.  Every pass must reproduce, bit for bit, the pass of the same inputs
run alone on one stream (parity of that pass with the oracle is covered by the other GPU tests);
passes in flight at the same time must not disturb each other."""
import numpy as np
import pytest
import torch

import gen
from gpu_harness import fetch, make_evaluator, upload
from paper_2603_02565_amd import flasheval as fe

pytestmark = pytest.mark.gpu

OUT = ("kv", "uniq", "n_uniq", "slot", "H", "seq", "Cp", "scores", "best")


def _inputs(c):
    """Two seeded input sets of one workload: the generated one, and the same with every
    request's lists reversed in order and its context rows (or ids) rolled by one."""
    I = gen.make_inputs(c)
    d0 = upload(c, I)
    d1 = dict(d0)
    d1["lists"] = torch.flip(d0["lists"], dims=[1]).contiguous()
    if d0["x"] is not None:
        d1["x"] = torch.roll(d0["x"], 1, dims=1).contiguous()
    else:
        d1["ctx_ids"] = torch.roll(d0["ctx_ids"], 1, dims=1).contiguous()
    return d0, d1


def _eager(ev, c, d):
    bufs = ev.allocate(c.B, c.T, c.M, c.K, c.L)
    ev.run(x=d["x"], ctx_ids=d["ctx_ids"], pool=d["pool"], lists=d["lists"], buffers=bufs)
    out = fetch(bufs)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("cid,kw,n_streams,n_pass", [
    (1, {}, 3, 7),                          # RecSys base, full batch
    (0, {}, 2, 5),                          # fp32 model
    (1, {"attention": "linear", "B": 8}, 3, 4),
    (4, {"B": 2, "T": 128, "K": 4}, 2, 3),  # token ids, d = 512 (tiled products)
])
def test_passes_in_flight_match_single_stream(cid, kw, n_streams, n_pass):
    c = gen.config(cid, **kw)
    W = gen.make_weights(c)
    ev = make_evaluator(c, W)
    d = _inputs(c)
    ref = [_eager(ev, c, d[0]), _eager(ev, c, d[1])]
    sets = [ev.allocate(c.B, c.T, c.M, c.K, c.L) for _ in range(n_streams)]
    for b in sets:                                   # outputs start as garbage
        for k in OUT:
            b[k].fill_(-7)
    ex = fe.Executor(ev, n_streams)
    last = {}
    for i in range(n_pass):
        k = i % n_streams
        di = d[i % 2]
        ex.submit(sets[k], x=di["x"], ctx_ids=di["ctx_ids"], pool=di["pool"], lists=di["lists"])
        last[k] = i % 2
    ex.join()
    torch.cuda.synchronize()
    print(f"\n[executor] {c.label}: {n_pass} passes over {n_streams} streams", flush=True)
    for k, which in last.items():
        got = fetch(sets[k])
        for name in OUT:
            assert np.array_equal(got[name], ref[which][name]), (c.label, k, name)
    ex.close()
    ev.close()


def test_graph_of_submissions_replays_exactly():
    """Three submissions and the join captured as one HIP graph (the executor's streams fork from
    and join the capturing stream): every replay, with eager passes on other inputs and cleared
    outputs between replays, reproduces the single-stream results."""
    c = gen.config(1, B=4)
    ev = make_evaluator(c, gen.make_weights(c))
    d0, d1 = _inputs(c)
    ref = [_eager(ev, c, d0), _eager(ev, c, d1)]
    sets = [ev.allocate(c.B, c.T, c.M, c.K, c.L) for _ in range(3)]
    ex = fe.Executor(ev, 3)
    feed = [d0, d1, d0]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        for k in range(3):
            ex.submit(sets[k], x=feed[k]["x"], pool=feed[k]["pool"], lists=feed[k]["lists"], stream=side)
        ex.join(side)
    torch.cuda.synchronize()
    for _ in range(3):
        ev.run(x=d1["x"], pool=d1["pool"], lists=d1["lists"], buffers=sets[0])   # eager work between replays
        torch.cuda.synchronize()
        for b in sets:
            for k in OUT:
                b[k].fill_(-7)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k in range(3):
            got = fetch(sets[k])
            want = ref[0] if feed[k] is d0 else ref[1]
            for name in OUT:
                assert np.array_equal(got[name], want[name]), (k, name)
    del graph
    ex.close()
    ev.close()


def test_submission_checked_before_anything_is_enqueued():
    c = gen.config(1, B=2, K=8)
    ev = make_evaluator(c, gen.make_weights(c))
    d = upload(c, gen.make_inputs(c))
    with pytest.raises(fe.FeError) as e:
        fe.Executor(ev, fe.FE_EXECUTOR_MAX_STREAMS + 1)
    assert e.value.status == fe.FE_EINVAL
    b = ev.allocate(c.B, c.T, c.M, c.K, c.L)
    b["scores"].fill_(-7)
    ex = fe.Executor(ev, 2)
    small = dict(b, ws=b["ws"][: b["ws"].numel() // 2])
    with pytest.raises(fe.FeError) as e:
        ex.submit(small, x=d["x"], pool=d["pool"], lists=d["lists"])
    assert e.value.status == fe.FE_EINVAL and "workspace" in str(e.value)
    with pytest.raises(fe.FeError) as e:
        ex.submit(b, x=d["x"], ctx_ids=torch.zeros((c.B, c.T), dtype=torch.int32, device="cuda"), pool=d["pool"],
                  lists=d["lists"])
    assert e.value.status == fe.FE_EINVAL
    ex.join()
    torch.cuda.synchronize()
    assert bool((b["scores"] == -7).all())           # nothing ran
    ex.close()
    ev.close()
