#!/usr/bin/env python3
"""Batched row-softmax bench on one MI355X.

A step is one pass of the whole hot path (plan lookup is built once, then every step launches
the persistent softmax kernel over the full batch: row loads, max, exp and sum, normalise,
store) over one batch of seeded synthetic input already resident in HBM. The headline workload
is BERT's attention-score shape: 384 slices of 512 x 512 fp32 packed as 196608 x 512.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c2] [--schedule xcd]

Prints ONE JSON line. `value` is achieved HBM GB/s with algorithmic bytes (every element read
once and written once) over the timed region; `roofline` reports the kernel's average launch
duration (HIP events on the launch stream) against the 8 TB/s HBM peak; `cpu_baseline` is the
fp64 oracle timed on this host's cores on the same workload.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "batched-softmax HBM GB/s (% of MI355X peak) at 384×512×512 fp32"
PEAK_HBM_GBS = 8000.0   # MI355X published HBM3E bandwidth
MALL_BYTES = 256 << 20  # last-level Infinity Cache; rotation keeps reuse distance above it


# device code of the kernel (launch wrappers excluded): a profile's counters stay valid while
# these files are unchanged
KERNEL_SOURCES = ("paper_2002_07062_amd/csrc/bsm_device.hpp", "paper_2002_07062_amd/csrc/bsm_tile.hpp")


def _kernel_sha() -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def _profiled(workload: str, schedule: str):
    """Figures of the committed rocprofv3 summary for this workload and schedule, and whether
    they were taken on the kernel as it is now (same source hash)."""
    path = os.path.join(ROOT, "profiles", f"bsm_softmax_kernel.{workload}.{schedule}.json")
    if not os.path.exists(path):
        return None, False
    with open(path) as fh:
        fig = json.load(fh)
    return fig, fig.get("kernel_sources_sha256") == _kernel_sha()


def _to_device(w):
    import numpy as np
    import torch

    if w.dtype == "f32":
        return torch.from_numpy(w.x).cuda()
    return torch.from_numpy(w.x.view(np.int16)).view(torch.bfloat16).cuda()


def _rotation(footprint: int) -> int:
    """Buffer pairs to rotate so the data a step touches was last used > 1 GB of traffic ago."""
    return max(2, math.ceil((4 * MALL_BYTES) / max(footprint, 1)) + 1)


def time_plan(plan, xs, outs, steps, warmup):
    """Returns (whole-region ms for `steps` back-to-back launches after `warmup`, per-launch ms
    of a separate pass). Only two events bracket the timed region, on the launch stream."""
    import torch

    import paper_2002_07062_amd as bsm

    n = len(xs)
    for i in range(warmup):
        bsm.bsm_plan_execute(plan, xs[i % n], outs[i % n])
    stream = torch.cuda.current_stream()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record(stream)
    for i in range(steps):
        bsm.bsm_plan_execute(plan, xs[i % n], outs[i % n])
    t1.record(stream)
    torch.cuda.synchronize()
    region = t0.elapsed_time(t1)
    # per-launch spread, outside the timed region (event records between launches add gaps)
    k = min(steps, 20)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(k)]
    for i in range(k):
        ev[i][0].record(stream)
        bsm.bsm_plan_execute(plan, xs[i % n], outs[i % n])
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    return region, [a.elapsed_time(b) for a, b in ev]


def time_copy(xs, outs, nbytes, steps, warmup):
    import torch

    import paper_2002_07062_amd as bsm

    n = len(xs)
    for i in range(warmup):
        bsm.bsm_copy(xs[i % n], outs[i % n], nbytes)
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record()
    for i in range(steps):
        bsm.bsm_copy(xs[i % n], outs[i % n], nbytes)
    t1.record()
    torch.cuda.synchronize()
    return t0.elapsed_time(t1) / steps


def run_workload(name, schedule, steps, warmup, rotate=None, w=None, topology=None,
                 xcd_weight=None):
    """Bench one (workload, schedule). Returns a dict of measurements."""
    import torch

    import paper_2002_07062_amd as bsm
    import workloads

    w = w or workloads.generate(name)
    nbytes = w.algorithmic_bytes
    n_pairs = rotate or _rotation(nbytes)
    x0 = _to_device(w)
    xs = [x0] + [x0.clone() for _ in range(n_pairs - 1)]
    outs = [torch.empty_like(x0) for _ in range(n_pairs)]
    t_plan = time.perf_counter()
    plan = bsm.bsm_plan_create(w.rows, w.cols, w.offsets[: w.batch], dtype=w.dtype,
                               schedule=schedule, topology=topology, device=0,
                               xcd_weight=xcd_weight)
    plan_ms = (time.perf_counter() - t_plan) * 1e3
    st = bsm.bsm_plan_describe(plan)
    region_ms, launch_ms = time_plan(plan, xs, outs, steps, warmup)
    plan.destroy()
    ms_step = region_ms / steps
    res = dict(
        workload=w.name, schedule=schedule, batch=w.batch, dtype=w.dtype,
        algorithmic_bytes=nbytes, ms_per_step=ms_step, gbs=nbytes / (ms_step * 1e-3) / 1e9,
        launch_ms_avg=ms_step, launch_ms_median=statistics.median(launch_ms),
        launch_ms_p10=sorted(launch_ms)[max(0, len(launch_ms) // 10 - 1)],
        launch_ms_p90=sorted(launch_ms)[min(len(launch_ms) - 1, (9 * len(launch_ms)) // 10)],
        launch_gbs=nbytes / (ms_step * 1e-3) / 1e9,
        slices_per_s=w.batch / (ms_step * 1e-3), plan_build_ms=plan_ms,
        n_wg=st["n_wg"], wg_threads=st["wg_threads"], n_items=st["n_items"],
        kernel_class=st["kernel_class"], n_workers=st["n_workers"], n_rounds=st["n_rounds"],
        max_over_mean_worker_cost=st["max_worker_cost"] / max(st["mean_worker_cost"], 1e-9),
        moved_bytes=st["moved_bytes"], buffers_rotated=n_pairs,
        lds_bytes_per_wave=st["lds_bytes_per_wave"])
    del xs, outs, x0
    torch.cuda.empty_cache()
    return res, w


def run_backward(name, schedule, steps, warmup, w=None):
    """Bench the backward op (dx from y and dy) on one workload: algorithmic bytes = every
    element of y and dy read once and dx written once. Inputs are the forward input itself
    and a seeded gradient: the kernel's work does not depend on the values."""
    import torch

    import paper_2002_07062_amd as bsm
    import workloads

    w = w or workloads.generate(name)
    nbytes = w.algorithmic_bytes * 3 // 2
    n_sets = _rotation(nbytes)
    y0 = _to_device(w)
    g = workloads.gradient(w)
    dy0 = (torch.from_numpy(g).cuda() if w.dtype == "f32"
           else torch.from_numpy(g.view("int16")).view(torch.bfloat16).cuda())
    ys = [y0] + [y0.clone() for _ in range(n_sets - 1)]
    dys = [dy0] + [dy0.clone() for _ in range(n_sets - 1)]
    dxs = [torch.empty_like(y0) for _ in range(n_sets)]
    plan = bsm.bsm_plan_create(w.rows, w.cols, w.offsets[: w.batch], dtype=w.dtype,
                               schedule=schedule, device=0)
    for i in range(warmup):
        bsm.bsm_plan_execute_backward(plan, ys[i % n_sets], dys[i % n_sets], dxs[i % n_sets])
    stream = torch.cuda.current_stream()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record(stream)
    for i in range(steps):
        bsm.bsm_plan_execute_backward(plan, ys[i % n_sets], dys[i % n_sets], dxs[i % n_sets])
    t1.record(stream)
    torch.cuda.synchronize()
    plan.destroy()
    ms = t0.elapsed_time(t1) / steps
    del ys, dys, dxs, y0, dy0
    torch.cuda.empty_cache()
    return dict(workload=w.name, schedule=schedule, algorithmic_bytes=nbytes, ms_per_step=ms,
                gbs=nbytes / (ms * 1e-3) / 1e9, buffers_rotated=n_sets)


GEMM_SHAPES = {  # Section 6's two batch products of BERT attention (batch, m, n, k, layout)
    "scores_384x512x512x64": (384, 512, 512, 64, "nt"),
    "context_384x512x64x512": (384, 512, 64, 512, "nn"),
    # the score product with the row softmax in the same kernel (P = softmax(Q K^T / 8))
    "scores_softmax_384x512x512x64": (384, 512, 512, 64, "nt_softmax"),
    # the same with a head dimension of 128 (one pass, A kept in LDS, two 64-deep chunks per step)
    "scores_softmax_192x512x512x128": (192, 512, 512, 128, "nt_softmax"),
}


def run_gemm(name, schedule, steps, warmup, out="bf16", topology=None):
    """Bench one batched product: algorithmic bytes = A and B read once + C written once;
    flops = 2 batch m n k."""
    import numpy as np
    import torch

    import paper_2002_07062_amd as bsm

    batch, m, n, k, layout = GEMM_SHAPES[name]
    es = 4 if out == "f32" else 2
    nbytes = batch * (2 * (m * k + n * k) + es * m * n)
    n_sets = _rotation(nbytes)
    rng = np.random.default_rng(5)
    a0 = torch.from_numpy(rng.standard_normal(batch * m * k, dtype=np.float32)).to(torch.bfloat16).cuda()
    b0 = torch.from_numpy(rng.standard_normal(batch * n * k, dtype=np.float32)).to(torch.bfloat16).cuda()
    tdt = torch.float32 if out == "f32" else torch.bfloat16
    As = [a0] + [a0.clone() for _ in range(n_sets - 1)]
    Bs = [b0] + [b0.clone() for _ in range(n_sets - 1)]
    Cs = [torch.empty(batch * m * n, dtype=tdt, device="cuda") for _ in range(n_sets)]
    plan = bsm.bsm_gemm_plan_create(batch, m, n, k, layout, out, schedule, topology=topology,
                                    device=0)
    for i in range(warmup):
        bsm.bsm_gemm_execute(plan, As[i % n_sets], Bs[i % n_sets], Cs[i % n_sets])
    stream = torch.cuda.current_stream()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record(stream)
    for i in range(steps):
        bsm.bsm_gemm_execute(plan, As[i % n_sets], Bs[i % n_sets], Cs[i % n_sets])
    t1.record(stream)
    torch.cuda.synchronize()
    plan.destroy()
    ms = t0.elapsed_time(t1) / steps
    del As, Bs, Cs, a0, b0
    torch.cuda.empty_cache()
    return dict(gbs=nbytes / (ms * 1e-3) / 1e9, tflops=2.0 * batch * m * n * k / (ms * 1e-3) / 1e12,
                ms_per_step=ms, algorithmic_bytes=nbytes, out=out)


def xcd_weight_calibration(name, steps, warmup):
    """Weighted load balancing (Section 4.2) with weights measured on this GPU: one traced
    launch of the unweighted XCD plan gives each XCD's rate (its bytes over the span of its
    waves); the weights are those rates (the inverse of each XCD's time per byte). Both plans
    are then timed."""
    import numpy as np
    import torch

    import paper_2002_07062_amd as bsm
    import workloads

    w = workloads.generate(name)
    x = _to_device(w)
    out = torch.empty_like(x)
    plan = bsm.bsm_plan_create(w.rows, w.cols, w.offsets[: w.batch], dtype=w.dtype,
                               schedule="xcd", device=0)
    st = bsm.bsm_plan_describe(plan)
    trace = torch.zeros(st["trace_bytes"], dtype=torch.uint8, device=x.device)
    rates = np.zeros(st["n_xcd"])
    for _ in range(3):  # average three traced launches
        bsm.bsm_plan_execute(plan, x, out)
        bsm.bsm_plan_execute(plan, x, out, trace=trace)
        torch.cuda.synchronize()
        rec = trace.cpu().numpy().view(bsm.TRACE_DTYPE)
        for xc in range(st["n_xcd"]):
            # the waves of the workers planned for XCD xc (workgroups w mod n_xcd == xc: the
            # bytes of xcd_bytes[xc]; dispatch may rotate which XCD runs them, uniformly)
            r = rec[rec["wg"] % st["n_xcd"] == xc]
            span = float(r["t_end"].max() - r["t_start"].min())
            rates[xc] += st["xcd_bytes"][xc] / max(span, 1.0)
    plan.destroy()
    del x, out, trace
    torch.cuda.empty_cache()
    weights = (rates / rates.max()).tolist()
    r0, _ = run_workload(name, "xcd", steps, warmup, w=w)
    r1, _ = run_workload(name, "xcd", steps, warmup, w=w, xcd_weight=weights)
    return {"weights": [round(v, 4) for v in weights], "unweighted_gbs": round(r0["gbs"], 1),
            "weighted_gbs": round(r1["gbs"], 1)}


def trace_stats(w, schedule):
    """One traced launch (outside any timed region): per-wave busy intervals from the kernel's
    constant-rate clock give the makespan, the mean wave busy time, the fraction of wave-time
    idle before the last wave ends, and the busiest XCD's time."""
    import numpy as np
    import torch

    import paper_2002_07062_amd as bsm

    hz = bsm.bsm_device_info(0)["wall_clock_hz"] or 100_000_000
    x = _to_device(w)
    out = torch.empty_like(x)
    plan = bsm.bsm_plan_create(w.rows, w.cols, w.offsets[: w.batch], dtype=w.dtype,
                               schedule=schedule, device=0)
    st = bsm.bsm_plan_describe(plan)
    trace = torch.zeros(st["trace_bytes"], dtype=torch.uint8, device=x.device)
    bsm.bsm_plan_execute(plan, x, out)  # warm
    bsm.bsm_plan_execute(plan, x, out, trace=trace)
    torch.cuda.synchronize()
    plan.destroy()
    rec = trace.cpu().numpy().view(bsm.TRACE_DTYPE)
    busy = (rec["t_end"] - rec["t_start"]).astype(np.float64) / hz * 1e6
    t0, t1 = int(rec["t_start"].min()), int(rec["t_end"].max())
    span = (t1 - t0) / hz * 1e6
    per_xcd, idle_xcd, start_xcd = {}, {}, {}
    for x_id in np.unique(rec["xcc_id"]):
        m = rec["xcc_id"] == x_id
        per_xcd[int(x_id)] = round(float((rec["t_end"][m].max() - t0) / hz * 1e6), 2)
        start_xcd[int(x_id)] = round(float((rec["t_start"][m].min() - t0) / hz * 1e6), 2)
        # wave-time of this XCD's waves left idle before the kernel's last wave ends
        idle_xcd[int(x_id)] = round(1.0 - float(busy[m].sum()) / (int(m.sum()) * span), 4) if span > 0 else 0.0
    working = rec["rows"] > 0
    n_xcd = max(1, int(st["n_xcd"]))
    rot = sorted(set(((rec["xcc_id"].astype(np.int64) - rec["wg"].astype(np.int64)) % n_xcd).tolist()))
    return {"makespan_us": round(span, 2), "mean_wave_busy_us": round(float(busy.mean()), 2),
            "idle_frac": round(1.0 - float(busy.sum()) / (len(busy) * span), 4) if span > 0 else 0.0,
            "waves_with_work": int(working.sum()), "waves": int(len(rec)),
            "xcd_finish_us": per_xcd, "xcd_first_start_us": start_xcd, "xcd_idle_frac": idle_xcd,
            "xcc_minus_wg_mod_n_xcd": rot}


def producer_consumer(iters=20):
    """Softmax right after a producer wrote its input (a device copy, standing in for the GEMM
    that computes attention scores), with the default streaming (nontemporal) accesses vs
    BSM_FLAG_TEMPORAL, at three batch sizes against the 256 MB Infinity Cache. Times the
    softmax launch only."""
    import torch

    import paper_2002_07062_amd as bsm
    import workloads

    cases = (("16MB", workloads.custom([512] * 16, [512] * 16, sigma=3.0, seed=4)),
             ("64MB", workloads.custom([512] * 64, [512] * 64, sigma=3.0, seed=4)),
             ("c3_201MB_bf16", workloads.generate("c3")))
    res = {}
    for name, w in cases:
        src = _to_device(w)
        x = torch.empty_like(src)
        out = torch.empty_like(src)
        row = {}
        for label, flags in (("streaming", 0), ("temporal", bsm.BSM_FLAG_TEMPORAL)):
            plan = bsm.bsm_plan_create(w.rows, w.cols, w.offsets[: w.batch], dtype=w.dtype,
                                       schedule="balanced", topology={"flags": flags}, device=0)
            ts = []
            for _ in range(iters):
                x.copy_(src)  # the producer
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                bsm.bsm_plan_execute(plan, x, out)
                e1.record()
                torch.cuda.synchronize()
                ts.append(e0.elapsed_time(e1))
            plan.destroy()
            row[label + "_us"] = round(statistics.median(ts) * 1e3, 2)
        res[name] = row
        del src, x, out
    return res


def attention_pipeline(steps=30, warmup=5, batch=384, seq=512, d=64):
    """Section 6's attention flow end to end, unfused: scores S = Q K^T / sqrt(d) (bf16 out),
    softmax of S in place (bf16), context O = P V (bf16 out), all under BALANCED, Q K V O rotated
    over enough sets to stay out of the Infinity Cache. Compares the default streaming
    (nontemporal) accesses with BSM_FLAG_TEMPORAL on all three plans, so that the 201 MB score
    tensor written by the first product can be served from the 256 MB Infinity Cache to the
    softmax and then to the second product. The "fused" variants compute P = softmax(Q K^T /
    sqrt(d)) in one kernel (the score product's "nt_softmax" layout: S never stored), then the
    context product, with streaming and with ordinary accesses. Returns microseconds per pipeline and per stage (each stage alone, same
    buffers) and algorithmic bytes."""
    import torch

    import paper_2002_07062_amd as bsm

    mk, ms = batch * seq * d, batch * seq * seq
    n_sets = max(2, math.ceil(4 * MALL_BYTES / (4 * mk * 2)) + 1)
    gen = torch.Generator(device="cuda").manual_seed(11)
    Q = [torch.randn(mk, device="cuda", generator=gen).bfloat16() for _ in range(n_sets)]
    K = [torch.randn(mk, device="cuda", generator=gen).bfloat16() for _ in range(n_sets)]
    V = [torch.randn(mk, device="cuda", generator=gen).bfloat16() for _ in range(n_sets)]
    O = [torch.empty(mk, device="cuda", dtype=torch.bfloat16) for _ in range(n_sets)]
    S = torch.empty(ms, device="cuda", dtype=torch.bfloat16)
    scale = 1.0 / math.sqrt(d)
    res = {"algorithmic_bytes": {"scores": batch * (2 * 2 * seq * d + 2 * seq * seq),
                                 "softmax": 2 * 2 * ms,
                                 "context": batch * (2 * seq * seq + 2 * seq * d + 2 * seq * d)}}

    def timed(fn):
        for i in range(warmup):
            fn(i % n_sets)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for i in range(steps):
            fn(i % n_sets)
        e1.record()
        torch.cuda.synchronize()
        return round(e0.elapsed_time(e1) / steps * 1e3, 2)

    for label, flags in (("streaming", 0), ("temporal", bsm.BSM_FLAG_TEMPORAL)):
        topo = {"flags": flags}
        p_s = bsm.bsm_gemm_plan_create(batch, seq, seq, d, "nt", "bf16", "balanced", topology=topo, device=0)
        p_c = bsm.bsm_gemm_plan_create(batch, seq, d, seq, "nn", "bf16", "balanced", topology=topo, device=0)
        p_m = bsm.bsm_plan_create([seq], [seq], None, dtype="bf16", schedule="balanced",
                                  topology=topo, device=0, batch=batch)

        def scores(i):
            bsm.bsm_gemm_execute(p_s, Q[i], K[i], S, scale)

        def soft(i):
            bsm.bsm_plan_execute(p_m, S, S)

        def context(i):
            bsm.bsm_gemm_execute(p_c, S, V[i], O[i])

        def pipe(i):
            scores(i)
            soft(i)
            context(i)

        res[label] = {"pipeline_us": timed(pipe), "scores_us": timed(scores),
                      "softmax_us": timed(soft), "context_us": timed(context)}
        for p in (p_s, p_c, p_m):
            p.destroy()
    # the score product and the softmax in one kernel, then the context product: streaming
    # accesses, and ordinary ones (P kept in the Infinity Cache for the context product)
    for label, flags in (("fused", 0), ("fused_temporal", bsm.BSM_FLAG_TEMPORAL)):
        topo = {"flags": flags}
        p_f = bsm.bsm_gemm_plan_create(batch, seq, seq, d, "nt_softmax", "bf16", "balanced",
                                       topology=topo, device=0)
        p_c = bsm.bsm_gemm_plan_create(batch, seq, d, seq, "nn", "bf16", "balanced", topology=topo,
                                       device=0)

        def probs(i):
            bsm.bsm_gemm_execute(p_f, Q[i], K[i], S, scale)

        def context_f(i):
            bsm.bsm_gemm_execute(p_c, S, V[i], O[i])

        def pipe_f(i):
            probs(i)
            context_f(i)

        res[label] = {"pipeline_us": timed(pipe_f), "scores_softmax_us": timed(probs),
                      "context_us": timed(context_f)}
        for p in (p_f, p_c):
            p.destroy()
    res["algorithmic_bytes"]["scores_softmax"] = res["algorithmic_bytes"]["scores"]
    del Q, K, V, O, S
    torch.cuda.empty_cache()
    return res


def l2_locality(nslices=16, iters=30):
    """Producer on each slice's home XCD, then the consumer on the same XCD or on the next one
    (XCD schedule with explicit homes), 16 MB working set: does the consumer find the
    producer's data in its XCD's L2 across the kernel boundary? Both policies."""
    import numpy as np
    import torch

    import paper_2002_07062_amd as bsm
    import workloads

    w = workloads.custom([512] * nslices, [512] * nslices, sigma=3.0, seed=3)
    x = _to_device(w)
    y, z = torch.empty_like(x), torch.empty_like(x)
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=x.device)
    home = (np.arange(nslices) % 8).astype(np.int8)
    res = {}
    for label, flags in (("streaming", 0), ("temporal", bsm.BSM_FLAG_TEMPORAL)):
        topo = {"flags": flags}
        mk = lambda h: bsm.bsm_plan_create(w.rows, w.cols, w.offsets[:-1], schedule="xcd",
                                           home_xcd=h, topology=topo, device=0)
        prod, same, skew = mk(home), mk(home), mk(((home + 1) % 8).astype(np.int8))
        ts = {"same_xcd": [], "next_xcd": [], "no_producer": []}
        for _ in range(iters):
            for k, plan in (("same_xcd", same), ("next_xcd", skew), ("no_producer", same)):
                flush.zero_()  # evict what the previous round left in the caches
                if k != "no_producer":
                    bsm.bsm_plan_execute(prod, x, y)
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                bsm.bsm_plan_execute(plan, y, z)
                e1.record()
                torch.cuda.synchronize()
                ts[k].append(e0.elapsed_time(e1) * 1e3)
        for p in (prod, same, skew):
            p.destroy()
        res[label] = {k: round(statistics.median(v), 2) for k, v in ts.items()}
    res["working_set_bytes"] = int(w.algorithmic_bytes // 2)
    return res


def time_hip_memcpy(xs, outs, nbytes, steps, warmup):
    """hipMemcpyAsync device-to-device of `nbytes` (the runtime's own copy engine path), same
    rotation and timing as time_copy: the vendor copy ceiling beside the library's copy kernel."""
    import ctypes

    import torch

    hip = ctypes.CDLL("libamdhip64.so.7")  # the runtime torch has loaded (same SONAME)
    hip.hipMemcpyAsync.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                   ctypes.c_int, ctypes.c_void_p]
    hip.hipMemcpyAsync.restype = ctypes.c_int
    dtod = 3  # hipMemcpyDeviceToDevice
    stream = torch.cuda.current_stream().cuda_stream
    n = len(xs)

    def cp(i):
        rc = hip.hipMemcpyAsync(outs[i % n].data_ptr(), xs[i % n].data_ptr(), nbytes, dtod, stream)
        if rc != 0:
            raise RuntimeError(f"hipMemcpyAsync failed ({rc})")

    for i in range(warmup):
        cp(i)
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record()
    for i in range(steps):
        cp(i)
    t1.record()
    torch.cuda.synchronize()
    return t0.elapsed_time(t1) / steps


def c3_balanced_bits(w):
    """One BALANCED launch on the bf16 workload `w`; returns the output's raw bf16 bits (host)."""
    import numpy as np
    import torch

    import paper_2002_07062_amd as bsm

    x = _to_device(w)
    out = torch.zeros_like(x)
    plan = bsm.bsm_plan_create(w.rows, w.cols, w.offsets[: w.batch], dtype=w.dtype,
                               schedule="balanced", device=0)
    bsm.bsm_plan_execute(plan, x, out)
    torch.cuda.synchronize()
    plan.destroy()
    bits = out.view(torch.int16).cpu().numpy().view(np.uint16)
    del x, out
    torch.cuda.empty_cache()
    return bits


def launch_bound_c1(steps=200, warmup=20):
    """C1 (8 slices of 64 x 64 fp32, 256 KiB): launch-bound, so the figure is microseconds per
    call. Per schedule: a plan's back-to-back executions (event-timed region / steps) and the
    host time of plan creation; and the one-shot call on a warm cache, called through the C ABI
    with its arguments marshalled once, and through the Python binding: host microseconds per
    call (argument checks, cache lookup, launch) and the event-timed region per call."""
    import ctypes

    import numpy as np
    import torch

    import paper_2002_07062_amd as bsm
    import workloads

    w = workloads.generate("c1")
    res = {"workload": w.name, "algorithmic_bytes": w.algorithmic_bytes}
    for sch in ("rr", "balanced", "xcd"):
        r, _ = run_workload("c1", sch, steps, warmup, rotate=2, w=w)
        res[sch] = {"us_per_call": round(r["ms_per_step"] * 1e3, 3),
                    "plan_build_ms": round(r["plan_build_ms"], 3), "n_items": r["n_items"]}
    x = _to_device(w)
    out = torch.empty_like(x)
    R, C = int(w.rows[0]), int(w.cols[0])
    lib = bsm.load()
    rows = np.array([R], np.int32)
    cols = np.array([C], np.int32)
    rp = rows.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    cp = cols.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    stream = torch.cuda.current_stream().cuda_stream
    xp, op = x.data_ptr(), out.data_ptr()

    def c_abi():
        rc = lib.bsm_softmax(xp, op, None, rp, cp, w.batch, bsm.BSM_F32, bsm.BSM_SCHED_BALANCED,
                             stream)
        if rc != bsm.BSM_OK:
            raise RuntimeError(bsm.bsm_last_error())

    def binding():
        bsm.bsm_softmax(x, out, R, C, batch=w.batch)

    for label, fn in (("one_shot_cached_c_abi", c_abi), ("one_shot_cached_python", binding)):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record()
        h0 = time.perf_counter()
        for _ in range(steps):
            fn()
        host = (time.perf_counter() - h0) / steps
        t1.record()
        torch.cuda.synchronize()
        res[label] = {"host_us_per_call": round(host * 1e6, 2),
                      "us_per_call": round(t0.elapsed_time(t1) / steps * 1e3, 3)}
    return res


def vendor_bmm(name, steps, warmup):
    """The same batched product through torch.bmm (hipBLASLt), bf16 operands and output,
    rotated like run_gemm; the scores product gets K already transposed and contiguous (bf16
    bmm of a transposed view is avoided). Times the product only; for the "nt_softmax" shape,
    the product followed by torch.softmax over each score row (the unfused library route)."""
    import numpy as np
    import torch

    batch, m, n, k, layout = GEMM_SHAPES[name]
    nbytes = batch * (2 * (m * k + n * k) + 2 * m * n)
    n_sets = _rotation(nbytes)
    rng = np.random.default_rng(5)
    a0 = torch.from_numpy(rng.standard_normal(batch * m * k, dtype=np.float32)).to(torch.bfloat16).cuda()
    b0 = torch.from_numpy(rng.standard_normal(batch * n * k, dtype=np.float32)).to(torch.bfloat16).cuda()
    A = [a0.view(batch, m, k)] + [a0.clone().view(batch, m, k) for _ in range(n_sets - 1)]
    if layout in ("nt", "nt_softmax"):  # B stored n x k per batch: hand bmm a k x n copy
        B = [b0.view(batch, n, k).transpose(1, 2).contiguous() for _ in range(n_sets)]
    else:
        B = [b0.view(batch, k, n)] + [b0.clone().view(batch, k, n) for _ in range(n_sets - 1)]
    Cs = [torch.empty(batch, m, n, dtype=torch.bfloat16, device="cuda") for _ in range(n_sets)]
    def run(i):
        torch.bmm(A[i], B[i], out=Cs[i])
        if layout == "nt_softmax":
            torch.softmax(Cs[i], dim=-1)

    for i in range(warmup):
        run(i % n_sets)
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record()
    for i in range(steps):
        run(i % n_sets)
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    del A, B, Cs, a0, b0
    torch.cuda.empty_cache()
    return {"us": round(ms * 1e3, 2), "gbs": round(nbytes / (ms * 1e-3) / 1e9, 1),
            "algorithmic_bytes": nbytes,
            "library": "torch.bmm (hipBLASLt)" + (" + torch.softmax" if layout == "nt_softmax" else "")}


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _bf16_rne_bits(v):
    """Round-to-nearest-even bf16 bit patterns of non-negative fp64 values (exact: the two bf16
    neighbours are compared in fp64; ties go to the even pattern)."""
    import numpy as np

    f = v.astype(np.float32)  # within 2^-24 of v: the bf16 neighbours of v are those of f
    lo = (f.view(np.uint32) >> 16).astype(np.uint32)
    hi = lo + 1
    lo_v = (lo << 16).view(np.float32).astype(np.float64)
    hi_v = (hi << 16).view(np.float32).astype(np.float64)
    d_lo, d_hi = v - lo_v, hi_v - v
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (lo % 2 == 1))
    return np.where(pick_hi, hi, lo).astype(np.uint16)


def cpu_baseline(w, bf16_check=None):
    """The fp64 oracle timed on this host: the whole workload at 1 thread and on all the
    threads this job may use (its affinity, capped at the 16 host threads a one-GPU job is
    given), repeated until 3 s have passed. bf16_check = (workload, GPU output bits): the oracle
    also runs on that bf16 workload (timed the same way, once), and the GPU outputs that are not
    the round-to-nearest-even bf16 of the fp64 value are counted."""
    import numpy as np

    import oracle

    avail = len(os.sched_getaffinity(0))
    share = min(16, avail)

    def timed(threads, min_s=3.0, work=w):
        out, reps = None, 0
        t0 = time.perf_counter()
        while reps < 1 or time.perf_counter() - t0 < min_s:
            out = oracle.softmax(work.x, work.dtype, work.offsets[: work.batch], work.rows,
                                 work.cols, nthreads=threads, out=out)
            reps += 1
        dt = (time.perf_counter() - t0) / reps
        return out, dt, reps

    _, dt, reps = timed(share)
    _, dt1, reps1 = timed(1)
    res = {"value": round(w.algorithmic_bytes / dt / 1e9, 3), "unit": "GB/s", "cores": share,
           "kind": "oracle", "seconds": round(dt * reps, 3),
           "sample": f"all {w.batch} slices of {w.name}, {reps} times (fp64 reference, {share} "
                     "threads, bytes counted as the fp32 read-once + write-once of the GPU path)",
           "single_thread": {"value": round(w.algorithmic_bytes / dt1 / 1e9, 3), "unit": "GB/s",
                             "cores": 1, "seconds": round(dt1 * reps1, 3),
                             "sample": f"all {w.batch} slices of {w.name}, {reps1} times"},
           "host_threads_in_affinity": avail, "cpu_model": _cpu_model()}
    if bf16_check is not None:
        wb, bits = bf16_check
        ref, dtb, _ = timed(share, 0.0, wb)
        live = ~np.isnan(ref)
        covered = np.zeros(ref.shape[0], bool)
        for o, R, C in zip(wb.offsets[: wb.batch], wb.rows, wb.cols):
            covered[int(o):int(o) + int(R) * int(C)] = True
        sel = live & covered
        non_rne = int(np.count_nonzero(bits[sel] != _bf16_rne_bits(ref[sel])))
        res["bf16_rounding"] = {
            "workload": wb.name, "outputs": int(sel.sum()), "non_rne": non_rne,
            "non_rne_frac": non_rne / max(1, int(sel.sum())),
            "oracle_seconds": round(dtb, 3),
            "note": "GPU bf16 outputs (BALANCED) that differ from the round-to-nearest-even "
                    "bf16 of the fp64 oracle value"}
    return res


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="c2")
    ap.add_argument("--schedule", default="balanced", choices=["rr", "balanced", "xcd"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true", help="headline line only")
    ap.add_argument("--op", default="forward", choices=["forward", "backward", "gemm"],
                    help="backward: time the gradient kernel alone on --workload and print its "
                         "line; gemm: time one batched product (--gemm, --out) alone (neither "
                         "is the headline metric)")
    ap.add_argument("--gemm", default="scores_384x512x512x64", choices=list(GEMM_SHAPES))
    ap.add_argument("--out", default="bf16", choices=["bf16", "f32"], help="--op gemm: C's type")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} (WORLD_SIZE {world}) is not "
              "supported: the batched softmax needs no exchange between GPUs, and the library "
              "runs on one MI355X at a time", file=sys.stderr)
        return 2

    import torch

    import paper_2002_07062_amd as bsm
    import workloads

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    bsm.load()
    info = bsm.bsm_device_info(0)

    if args.op == "backward":
        # the backward op alone, with the copy reference for the counters' scale factors
        r = run_backward(args.workload, args.schedule, args.steps, args.warmup)
        wb = workloads.generate(args.workload)
        x0 = _to_device(wb)
        n_pairs = _rotation(wb.algorithmic_bytes)
        xs = [x0] + [x0.clone() for _ in range(n_pairs - 1)]
        outs = [torch.empty_like(x0) for _ in range(n_pairs)]
        copy_ms = time_copy(xs, outs, wb.algorithmic_bytes // 2, args.steps, args.warmup)
        print(json.dumps({
            "metric": "batched-softmax backward HBM GB/s (read y and dy, write dx)",
            "value": round(r["gbs"], 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": round(r["ms_per_step"], 5),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
            "dtype": wb.dtype, "data": "synthetic",
            "config": {"workload": wb.name, "schedule": args.schedule, "op": "backward"},
            "pct_of_peak": round(100 * r["gbs"] / PEAK_HBM_GBS, 2),
            "algorithmic_bytes": r["algorithmic_bytes"],
            "copy_reference_gbs": round(wb.algorithmic_bytes / (copy_ms * 1e-3) / 1e9, 1)}))
        return 0

    if args.op == "gemm":
        # one batched product alone, with the copy reference (half the bytes each way) for
        # the counters' scale factors
        r = run_gemm(args.gemm, args.schedule, args.steps, args.warmup, out=args.out)
        batch, m, n, k, layout = GEMM_SHAPES[args.gemm]
        half = r["algorithmic_bytes"] // 2 // 16 * 16
        n_pairs = _rotation(2 * half)
        xs = [torch.empty(half // 4, device="cuda") for _ in range(n_pairs)]
        outs = [torch.empty_like(x) for x in xs]
        copy_ms = time_copy(xs, outs, half, args.steps, args.warmup)
        print(json.dumps({
            "metric": f"batched matrix product HBM GB/s ({args.gemm}, {layout}, bf16 in, {args.out} out)",
            "value": round(r["gbs"], 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": round(r["ms_per_step"], 5),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
            "dtype": "bf16", "data": "synthetic",
            "config": {"workload": args.gemm, "batch": batch, "m": m, "n": n, "k": k,
                       "layout": layout, "out": args.out, "schedule": args.schedule, "op": "gemm"},
            "tflops": round(r["tflops"], 2), "pct_of_peak": round(100 * r["gbs"] / PEAK_HBM_GBS, 2),
            "algorithmic_bytes": r["algorithmic_bytes"], "copy_bytes_each_way": half,
            "copy_reference_gbs": round(2 * half / (copy_ms * 1e-3) / 1e9, 1)}))
        return 0

    head, w = run_workload(args.workload, args.schedule, args.steps, args.warmup)

    # Copy ceiling on the same bytes (read n/2, write n/2), same rotation.
    import numpy as np  # noqa: F401

    x0 = _to_device(w)
    n_pairs = head["buffers_rotated"]
    xs = [x0] + [x0.clone() for _ in range(n_pairs - 1)]
    outs = [torch.empty_like(x0) for _ in range(n_pairs)]
    half = w.algorithmic_bytes // 2
    copy_ms = time_copy(xs, outs, half, args.steps, args.warmup)
    memcpy_ms = time_hip_memcpy(xs, outs, half, args.steps, args.warmup)
    del xs, outs, x0
    torch.cuda.empty_cache()
    copy_gbs = w.algorithmic_bytes / (copy_ms * 1e-3) / 1e9
    memcpy_gbs = w.algorithmic_bytes / (memcpy_ms * 1e-3) / 1e9

    extra = {}
    if not args.no_extra:
        for sch in ("rr", "balanced", "xcd"):
            if sch == args.schedule:
                continue
            r, _ = run_workload(args.workload, sch, args.steps, args.warmup, w=w)
            extra[f"{args.workload}_{sch}"] = {k: r[k] for k in ("gbs", "launch_ms_avg", "ms_per_step", "max_over_mean_worker_cost", "plan_build_ms")}
        for sch in ("rr", "balanced", "xcd"):
            if sch != args.schedule:
                extra[f"{args.workload}_{sch}"]["trace"] = trace_stats(w, sch)
        for cfg in ("c3", "c4", "c5"):
            wk = None
            for sch in ("rr", "balanced", "xcd"):
                r, wk = run_workload(cfg, sch, args.steps, args.warmup, w=wk)
                extra[f"{cfg}_{sch}"] = {k: r[k] for k in ("gbs", "ms_per_step", "max_over_mean_worker_cost",
                                                        "moved_bytes", "n_items", "plan_build_ms")}
                if cfg in ("c4", "c5"):
                    extra[f"{cfg}_{sch}"]["trace"] = trace_stats(wk, sch)
                if cfg == "c3" and sch == "balanced":
                    c3_bits = c3_balanced_bits(wk)
            del wk
        extra["c1"] = launch_bound_c1()
        # one GPU's share of C2 under 8-way head sharding: 48 slices, where a slice per
        # workgroup can occupy at most 48 of the 512 workgroups
        wk = workloads.generate("c2", batch=48)
        for sch in ("rr", "balanced", "xcd"):
            r, _ = run_workload("c2", sch, args.steps, args.warmup, w=wk)
            extra[f"shard8_48x512x512_f32_{sch}"] = {k: r[k] for k in ("gbs", "ms_per_step", "n_items")}
        del wk
        # the backward op (dx = y * (dy - sum(dy * y))): three streams, same tables
        for cfg, sch in (("c2", "balanced"), ("c2", "xcd"), ("c2", "rr"), ("c3", "balanced"),
                         ("c5", "balanced"), ("c5", "rr")):
            r = run_backward(cfg, sch, args.steps, args.warmup)
            extra[f"{cfg}_backward_{sch}"] = {k: r[k] for k in ("gbs", "ms_per_step", "algorithmic_bytes")}
        extra["xcd_weighted_c2"] = xcd_weight_calibration("c2", args.steps, args.warmup)
        # Section 6's batch products around the softmax, bf16 in and out, per schedule
        for gname in GEMM_SHAPES:
            res = {sch: run_gemm(gname, sch, args.steps, args.warmup) for sch in ("rr", "balanced", "xcd")}
            extra[f"gemm_{gname}"] = {sch: {k: round(v, 4) if isinstance(v, float) else v
                                            for k, v in r.items()} for sch, r in res.items()}
            extra[f"gemm_{gname}"]["balanced_over_rr"] = round(res["rr"]["ms_per_step"] /
                                                               res["balanced"]["ms_per_step"], 3)
            extra[f"gemm_{gname}"]["vendor"] = vendor_bmm(gname, args.steps, args.warmup)
        extra["producer_consumer"] = producer_consumer()
        extra["attention_pipeline"] = attention_pipeline()
        extra["l2_locality_16MB_us"] = l2_locality()
        # rows longer than the register tile, held in the registers of a workgroup (256 threads:
        # up to 8192 elements in kernel class 4, 16384 in class 5; 512 threads: up to 32768 in
        # class 6) and read once, forward and backward
        for name in ("long4k", "long", "long16k", "long32k", "long4104bf16", "long8200bf16"):
            r, _ = run_workload(name, "balanced", args.steps, args.warmup)
            extra[f"{name}_balanced"] = {k: r[k] for k in ("gbs", "ms_per_step", "kernel_class")}
            r = run_backward(name, "balanced", args.steps, args.warmup)
            extra[f"{name}_backward_balanced"] = {k: r[k] for k in ("gbs", "ms_per_step")}
        # uniform fp32 batches at one row width each: full and partly filled register tiles
        extra["widths_f32"] = {}
        for c in (64, 72, 96, 136, 264, 520):
            r, _ = run_workload(f"w{c}", "balanced", args.steps, args.warmup)
            rb = run_backward(f"w{c}", "balanced", args.steps, args.warmup)
            extra["widths_f32"][str(c)] = {"gbs": round(r["gbs"], 1),
                                           "backward_gbs": round(rb["gbs"], 1),
                                           "ms_per_step": r["ms_per_step"]}
        # rows that do not start or end on a 16-byte vector (1001 fp32): shifted vectors
        r, _ = run_workload("odd", "balanced", args.steps, args.warmup)
        extra["odd_balanced"] = {k: r[k] for k in ("gbs", "ms_per_step", "kernel_class")}
        r = run_backward("odd", "balanced", args.steps, args.warmup)
        extra["odd_backward_balanced"] = {k: r[k] for k in ("gbs", "ms_per_step")}

    head_trace = None if args.no_extra else trace_stats(w, args.schedule)
    cpu = None
    if not args.no_cpu_baseline:
        check = None
        if not args.no_extra:
            check = (workloads.generate("c3"), c3_bits)
        cpu = cpu_baseline(w, check)
    achieved = head["launch_gbs"]
    prof, current = _profiled(head["workload"], args.schedule)
    line = {
        "metric": METRIC,
        "value": round(head["gbs"], 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(head["ms_per_step"], 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if w.dtype == "f32" else "bf16",
        "data": "synthetic",
        "config": {"workload": head["workload"], "batch": head["batch"],
                   "rows": int(w.rows[0]) if w.uniform else "ragged",
                   "cols": int(w.cols[0]) if w.uniform else "ragged",
                   "schedule": args.schedule, "n_wg": head["n_wg"],
                   "wg_threads": head["wg_threads"], "n_workers": head["n_workers"],
                   "n_rounds": head["n_rounds"], "buffers_rotated": head["buffers_rotated"]},
        "pct_of_peak": round(100.0 * head["gbs"] / PEAK_HBM_GBS, 2),
        "slices_per_s": round(head["slices_per_s"], 1),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4),
                     "traffic": prof["traffic_bytes_per_launch"] if (prof and current) else None,
                     "traffic_over_algorithmic": round(prof["traffic_over_algorithmic"], 5) if (prof and current) else None,
                     "rocprof_avg_us": round(prof["avg_ns"] / 1e3, 2) if (prof and current) else None,
                     "kernel": "bsm_softmax_kernel",
                     "launch_us_avg": round(head["launch_ms_avg"] * 1e3, 2),
                     "launch_us_median_single": round(head["launch_ms_median"] * 1e3, 2),
                     "launch_us_p10_single": round(head["launch_ms_p10"] * 1e3, 2),
                     "launch_us_p90_single": round(head["launch_ms_p90"] * 1e3, 2),
                     "bytes_per_launch": head["algorithmic_bytes"],
                     "profile": (f"profiles/bsm_softmax_kernel.{head['workload']}.{args.schedule}.json: "
                                 "rocprofv3 summary committed with the kernel source it was taken "
                                 "on (same sha256 as now), on another MI355X of the same kind"
                                 if (prof and current) else None)},
        "trace": head_trace,
        "copy_ceiling": {"gbs": round(copy_gbs, 2), "us": round(copy_ms * 1e3, 2),
                         "softmax_pct_of_copy": round(100.0 * head["gbs"] / copy_gbs, 2),
                         "hipMemcpyAsync_dtod_gbs": round(memcpy_gbs, 2),
                         "hipMemcpyAsync_dtod_us": round(memcpy_ms * 1e3, 2),
                         "softmax_pct_of_hipMemcpyAsync": round(100.0 * head["gbs"] / memcpy_gbs, 2)},
        "plan_build_ms": round(head["plan_build_ms"], 3),
        "cpu_baseline": cpu,
        "device": {"arch": info["arch"], "n_cu": info["n_cu"], "n_xcd": info["n_xcd"]},
        "extra": extra,
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
