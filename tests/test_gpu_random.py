"""Randomized parity on the GPU: seeded random geometries (slices in random order with gaps,
empty slices, widths 1 ... 9000 across every kernel class) through all three schedules against
the fp64 oracle, forward and backward, and random batched-product shapes (tails in every
dimension, k = 0 included) against the product oracle. Every schedule must also give the same
bits as the others."""

import numpy as np
import pytest
import torch

import oracle
import paper_2002_07062_amd as bsm
import workloads
from gpu_util import (SENTINEL_BF16, SENTINEL_F32, backward_inputs, compare, compare_backward,
                      covered_mask, run_plan, run_plan_backward, to_device, to_host_bits)
from oracle import gemm as og
from random_geometry import geometry

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("seed", range(12))
def test_random_geometries_forward_all_schedules(seed):
    dtype = "f32" if seed % 2 == 0 else "bf16"
    w = geometry(100 + seed, max_batch=30, max_rows=60, dtype=dtype)
    print(f"[random fwd seed {seed} {dtype} batch {w.batch} max_cols {int(w.cols.max()) if w.batch else 0}]", flush=True)
    n = int(w.offsets[-1])
    ref = oracle.softmax(w.x, w.dtype, w.offsets[: w.batch], w.rows, w.cols, nthreads=16)
    mask = covered_mask(w.offsets[: w.batch], w.rows, w.cols, n)
    x = to_device(w.x, w.dtype)
    first = None
    for schedule in ("rr", "balanced", "xcd"):
        out, _ = run_plan(w, schedule, x=x)
        bits = to_host_bits(out)
        if n:
            compare(bits[:n], ref, w.dtype, mask)
            sentinel = SENTINEL_F32 if dtype == "f32" else SENTINEL_BF16
            assert np.all(bits[:n][~mask] == sentinel), "a byte outside every slice was written"
        if first is None:
            first = bits
        else:
            assert np.array_equal(bits, first), schedule


@pytest.mark.parametrize("seed", range(6))
def test_random_geometries_backward(seed):
    dtype = "f32" if seed % 2 == 0 else "bf16"
    w = geometry(200 + seed, max_batch=24, max_rows=40, dtype=dtype)
    if w.batch == 0 or int(w.offsets[-1]) == 0:
        pytest.skip("empty geometry")
    print(f"[random bwd seed {seed} {dtype} batch {w.batch}]", flush=True)
    n = int(w.offsets[-1])
    y, dy = backward_inputs(w)
    ref = oracle.softmax_backward(y, dy, w.dtype, w.offsets[: w.batch], w.rows, w.cols, nthreads=16)
    mask = covered_mask(w.offsets[: w.batch], w.rows, w.cols, n)
    yd, dyd = to_device(y, w.dtype), to_device(dy, w.dtype)
    first = None
    for schedule in ("rr", "balanced", "xcd"):
        dx, _ = run_plan_backward(w, yd, dyd, schedule)
        bits = to_host_bits(dx)
        compare_backward(bits, ref, y, dy, w.dtype, w.offsets[: w.batch], w.rows, w.cols, mask)
        if first is None:
            first = bits
        else:
            assert np.array_equal(bits, first), schedule


@pytest.mark.parametrize("seed", range(10))
def test_random_product_shapes(seed):
    rng = np.random.default_rng(300 + seed)
    batch = int(rng.integers(1, 7))
    m, n = (int(v) for v in rng.integers(1, 300, size=2))
    k = int(rng.choice([0, 1, 8, 24, 64, 72, 130, 300]))
    layout = str(rng.choice(["nt", "nn"]))
    out = str(rng.choice(["f32", "bf16"]))
    print(f"[random gemm seed {seed}: batch {batch} m {m} n {n} k {k} {layout} {out}]", flush=True)
    a = workloads._to_bf16_bits(rng.standard_normal(batch * m * k, dtype=np.float32))
    b = workloads._to_bf16_bits(rng.standard_normal(batch * n * k, dtype=np.float32))
    a_d = torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda() if k else torch.zeros(8, dtype=torch.bfloat16, device="cuda")
    b_d = torch.from_numpy(b.view(np.int16)).view(torch.bfloat16).cuda() if k else torch.zeros(8, dtype=torch.bfloat16, device="cuda")
    tdt = torch.float32 if out == "f32" else torch.bfloat16
    ref = og.batched_gemm(a, b, batch, m, n, k, layout, 0.5) if k else np.zeros(batch * m * n)
    bound = (2.0 * max(k, 1) * 2.0 ** -24 * 0.5 * og.abs_product_sums(a, b, batch, m, n, k, layout)
             if k else np.zeros(batch * m * n))
    if out == "bf16":
        bound = 2.0 ** -8 * np.abs(ref) + 2.0 * bound
    first = None
    for schedule in ("rr", "balanced", "xcd"):
        c = torch.full((batch * m * n + 3,), float("nan"), dtype=tdt, device="cuda")
        p = bsm.bsm_gemm_plan_create(batch, m, n, k, layout, out, schedule, device=0)
        bsm.bsm_gemm_execute(p, a_d, b_d, c, 0.5)
        torch.cuda.synchronize()
        p.destroy()
        got = c.float().cpu().numpy().astype(np.float64)
        assert np.all(np.abs(got[: batch * m * n] - ref) <= bound), schedule
        assert np.all(np.isnan(got[batch * m * n:])), "written past C"
        bits = to_host_bits(c)
        if first is None:
            first = bits
        else:
            assert np.array_equal(bits, first), schedule
