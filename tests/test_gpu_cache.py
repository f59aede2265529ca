"""The one-shot calls' plan cache on the GPU: no call waits for the device (misses upload their
table asynchronously and evictions free nothing), a warm call captured in a HIP graph replays
correctly, a miss under capture is refused cleanly, and a failed device allocation reports
BSM_ERR_OOM and leaves the library usable. Oracle: the fp64 CPU reference."""

import time

import numpy as np
import pytest
import torch

import oracle
import paper_2002_07062_amd as bsm
import workloads
from gpu_util import compare, sentinel_like, to_device, to_host_bits

pytestmark = pytest.mark.gpu


def _cases(n, seed):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        B = int(rng.integers(1, 6))
        R = int(rng.integers(1, 9))
        C = int(rng.integers(8, 700))
        out.append((B, R, C))
    return out


def test_one_shot_calls_never_wait_for_the_device():
    """40 geometries (more than the 32 the cache keeps, so every call after the first pass is a
    miss that evicts) cycled twice over two streams, each stream holding a long queue of copies
    enqueued first. Every call returns while both queues are still running -- a call that built
    a plan, uploaded a table, evicted or reused a buffer never waited for the device -- and
    after the queues drain every output matches the oracle."""
    bsm.bsm_cache_clear()
    cases = _cases(40, 31)
    xs, refs = [], []
    for B, R, C in cases:
        w = workloads.custom([R] * B, [C] * B, sigma=2.0, seed=B * 1000 + C)
        xs.append(to_device(w.x, "f32"))
        refs.append(oracle.softmax(w.x, "f32", w.offsets[:-1], w.rows, w.cols))
    outs = [[sentinel_like(x.numel(), "f32") for x in xs] for _ in range(2)]
    # warm the library (kernel code objects load on first launch)
    warm = torch.zeros(4096, device="cuda")
    bsm.bsm_softmax(warm, warm, 4, 1024, batch=1)
    n_big = 1 << 28  # 1 GiB of fp32 per buffer
    src = torch.zeros(n_big, device="cuda")
    dst = [torch.empty(n_big, device="cuda") for _ in range(2)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    reps = 400  # ~2 GiB of traffic per copy: the two queues hold a few hundred ms of work
    for s, d in zip(streams, dst):
        with torch.cuda.stream(s):
            for _ in range(reps):
                bsm.bsm_copy(src, d)
    t0 = time.perf_counter()
    per_call = []
    for rep in range(2):
        for i, (B, R, C) in enumerate(cases):
            s = streams[(i + rep) % 2]
            t = time.perf_counter()
            with torch.cuda.stream(s):
                bsm.bsm_softmax(xs[i], outs[rep][i], R, C, batch=B,
                                schedule=("rr", "balanced", "xcd")[i % 3])
            per_call.append(time.perf_counter() - t)
    host = time.perf_counter() - t0
    busy = [not s.query() for s in streams]
    t1 = time.perf_counter()
    torch.cuda.synchronize()
    drain = time.perf_counter() - t1
    print(f"80 one-shot calls: host {host * 1e3:.1f} ms (max per call "
          f"{max(per_call) * 1e6:.0f} us, median {np.median(per_call) * 1e6:.0f} us); "
          f"queues still busy {busy}, drained {drain * 1e3:.1f} ms later", flush=True)
    assert all(busy), "a one-shot call waited for the device"
    assert host < drain, (host, drain)
    for rep in range(2):
        for i in range(len(cases)):
            compare(to_host_bits(outs[rep][i]), refs[i], "f32")
    del src, dst
    bsm.bsm_cache_clear()


def test_warm_one_shot_call_replays_from_a_captured_graph():
    """A one-shot call whose plan is cached can be captured: the replays (new inputs written
    eagerly between them) match eager calls bit for bit and the oracle, and the captured plan
    survives more than 32 other geometries passing through the cache. A geometry not in the
    cache is refused under capture with BSM_ERR_UNSUPPORTED, and the capture goes on."""
    bsm.bsm_cache_clear()
    w = workloads.custom([6, 3, 9], [512, 1000, 72], sigma=3.0, seed=71, gap=4)
    n = int(w.offsets[-1])
    x = to_device(w.x, "f32")
    out = torch.zeros_like(x)
    other = to_device(workloads.custom([2], [64], seed=72).x, "f32")
    other_out = torch.zeros_like(other)
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):  # warm: the miss, then a hit that sees the upload done
        bsm.bsm_softmax(x, out, w.rows, w.cols, slice_offsets=w.offsets[:-1])
        stream.synchronize()
        bsm.bsm_softmax(x, out, w.rows, w.cols, slice_offsets=w.offsets[:-1])
    stream.synchronize()
    graph = torch.cuda.CUDAGraph()
    refused = None
    with torch.cuda.graph(graph, stream=stream):
        bsm.bsm_softmax(x, out, w.rows, w.cols, slice_offsets=w.offsets[:-1])
        try:
            bsm.bsm_softmax(other, other_out, 2, 64, batch=1, schedule="xcd")
        except bsm.BsmError as e:
            refused = e
    assert refused is not None and refused.status == bsm.BSM_ERR_UNSUPPORTED, refused
    assert "capture" in refused.message
    # push more than the cache's 32 geometries through it: the captured plan stays
    for B, R, C in _cases(40, 73):
        t = torch.zeros(B * R * C, device="cuda")
        bsm.bsm_softmax(t, t, R, C, batch=B)
    torch.cuda.synchronize()
    rng = np.random.default_rng(74)
    for rep in range(4):
        print(f"[one-shot graph replay {rep}]", flush=True)
        xv = (rng.standard_normal(n) * 3).astype(np.float32)
        x.copy_(torch.from_numpy(xv).cuda())
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        eager = torch.zeros_like(x)
        bsm.bsm_softmax(x, eager, w.rows, w.cols, slice_offsets=w.offsets[:-1])
        torch.cuda.synchronize()
        bits = to_host_bits(out)
        assert np.array_equal(bits, to_host_bits(eager)), rep
        ref = oracle.softmax(xv, "f32", w.offsets[:-1], w.rows, w.cols)
        from gpu_util import covered_mask
        compare(bits, ref, "f32", covered_mask(w.offsets[:-1], w.rows, w.cols, n))
    del graph
    bsm.bsm_cache_clear()


def test_device_allocation_failure_reports_oom_and_recovers(monkeypatch):
    """With the test hook BSM_TEST_ALLOC_FAIL=device the work table's device allocation fails:
    a one-shot call (cache miss) and a plan creation both return BSM_ERR_OOM with a message and
    launch nothing (the output keeps its sentinel); without the hook the same calls succeed and
    match the oracle."""
    bsm.bsm_cache_clear()
    w = workloads.custom([4, 4], [256, 256], sigma=2.0, seed=81)
    x = to_device(w.x, "f32")
    out = sentinel_like(x.numel(), "f32")
    monkeypatch.setenv("BSM_TEST_ALLOC_FAIL", "device")
    with pytest.raises(bsm.BsmError) as e1:
        bsm.bsm_softmax(x, out, w.rows, w.cols, slice_offsets=w.offsets[:-1])
    assert e1.value.status == bsm.BSM_ERR_OOM and "hipMalloc" in e1.value.message
    with pytest.raises(bsm.BsmError) as e2:
        bsm.bsm_plan_create(w.rows, w.cols, w.offsets[:-1], dtype="f32", device=0)
    assert e2.value.status == bsm.BSM_ERR_OOM
    torch.cuda.synchronize()
    assert np.all(to_host_bits(out) == np.uint32(0x7FC0DEAD))
    monkeypatch.delenv("BSM_TEST_ALLOC_FAIL")
    ref = oracle.softmax(w.x, "f32", w.offsets[:-1], w.rows, w.cols)
    bsm.bsm_softmax(x, out, w.rows, w.cols, slice_offsets=w.offsets[:-1])
    plan = bsm.bsm_plan_create(w.rows, w.cols, w.offsets[:-1], dtype="f32", device=0)
    out2 = sentinel_like(x.numel(), "f32")
    bsm.bsm_plan_execute(plan, x, out2)
    torch.cuda.synchronize()
    plan.destroy()
    compare(to_host_bits(out), ref, "f32")
    compare(to_host_bits(out2), ref, "f32")
    bsm.bsm_cache_clear()
