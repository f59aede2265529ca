"""Helpers for the GPU parity tests: upload seeded inputs, run the HIP path through the C ABI,
compare with the fp64 oracle at the stated tolerances."""

from __future__ import annotations

import numpy as np
import torch

import oracle
import paper_2002_07062_amd as bsm

F32_ATOL = 2e-6          # max abs error for fp32 outputs
BF16_REL = 2.0 ** -8     # |y - y_ref| <= 2^-8 |y_ref| for bf16 outputs

SENTINEL_F32 = np.uint32(0x7FC0DEAD)  # a NaN payload no computation produces
SENTINEL_BF16 = np.uint16(0x7FDE)


def dev():
    return torch.device("cuda", 0)


def to_device(x: np.ndarray, dtype: str, pad: int = 0) -> torch.Tensor:
    """Flat input on the GPU (bf16 bit patterns become a bfloat16 tensor)."""
    if dtype == "f32":
        t = torch.from_numpy(np.ascontiguousarray(x, np.float32))
    else:
        t = torch.from_numpy(np.ascontiguousarray(x, np.uint16).view(np.int16)).view(torch.bfloat16)
    if pad:
        t = torch.cat([t, torch.zeros(pad, dtype=t.dtype)])
    return t.to(dev())


def sentinel_like(n: int, dtype: str) -> torch.Tensor:
    if dtype == "f32":
        a = np.full(n, SENTINEL_F32, np.uint32).view(np.float32)
        return torch.from_numpy(a).to(dev())
    a = np.full(n, SENTINEL_BF16, np.uint16).view(np.int16)
    return torch.from_numpy(a).view(torch.bfloat16).to(dev())


def to_host_bits(t: torch.Tensor) -> np.ndarray:
    """Raw bits of a GPU tensor (uint32 for fp32, uint16 for bf16)."""
    if t.dtype == torch.float32:
        return t.cpu().numpy().view(np.uint32)
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def bits_to_f64(bits: np.ndarray) -> np.ndarray:
    if bits.dtype == np.uint32:
        return bits.view(np.float32).astype(np.float64)
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def covered_mask(offsets, rows, cols, n: int) -> np.ndarray:
    m = np.zeros(n, bool)
    for o, R, C in zip(offsets, rows, cols):
        m[int(o):int(o) + int(R) * int(C)] = True
    return m


def compare(y_bits: np.ndarray, y_ref: np.ndarray, dtype: str, mask: np.ndarray | None = None):
    """Checks the GPU result against the fp64 oracle on `mask` (default: everywhere).
    Returns (max_abs_err, n_checked)."""
    y = bits_to_f64(y_bits)
    if mask is not None:
        y, y_ref = y[mask], y_ref[mask]
    nan_ref = np.isnan(y_ref)
    assert np.array_equal(np.isnan(y), nan_ref), "NaN positions differ"
    y, y_ref = y[~nan_ref], y_ref[~nan_ref]
    err = np.abs(y - y_ref)
    if dtype == "f32":
        bad = err > F32_ATOL
        assert not bad.any(), f"{int(bad.sum())} fp32 outputs beyond {F32_ATOL}: max {err.max():.3e}"
    else:
        bad = err > BF16_REL * np.abs(y_ref)
        assert not bad.any(), (f"{int(bad.sum())} bf16 outputs beyond 2^-8 relative; "
                               f"worst {err[bad].max():.3e} at ref {y_ref[bad][np.argmax(err[bad])]:.3e}")
        zero = y_ref == 0.0
        ybits = y_bits[mask][~nan_ref] if mask is not None else y_bits[~nan_ref]
        assert np.all(ybits[zero] == 0), "an exact-zero reference did not give +0"
    return (float(err.max()) if err.size else 0.0), int(y.size)


def bf16_rne_bits(v: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even bf16 bit patterns of non-negative fp64 values: the two bf16
    neighbours of v (those of its nearest fp32, which lies within half an fp32 ulp of v, never
    across a bf16 value) compared in fp64, ties to the even pattern."""
    f = v.astype(np.float32)
    lo = (f.view(np.uint32) >> 16).astype(np.uint32)
    hi = lo + 1
    lo_v = (lo << 16).view(np.float32).astype(np.float64)
    hi_v = (hi << 16).view(np.float32).astype(np.float64)
    d_lo, d_hi = v - lo_v, hi_v - v
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (lo % 2 == 1))
    return np.where(pick_hi, hi, lo).astype(np.uint16)


def count_non_rne(y_bits: np.ndarray, y_ref: np.ndarray) -> tuple[int, int]:
    """bf16 outputs that are not the round-to-nearest-even of the fp64 reference (NaN rows
    excluded): (count, outputs compared)."""
    live = ~np.isnan(y_ref)
    return int(np.count_nonzero(y_bits[live] != bf16_rne_bits(y_ref[live]))), int(live.sum())


def run_plan(w, schedule="xcd", x=None, out=None, topology=None, trace=None, home_xcd=None):
    """Run the workload through bsm_plan_create/execute; returns (out tensor, plan stats)."""
    offsets = w.offsets[: w.batch]
    n = int(w.offsets[-1]) if len(w.offsets) else 0
    if x is None:
        x = to_device(w.x, w.dtype)
    if out is None:
        out = sentinel_like(max(n, 1), w.dtype)
    plan = bsm.bsm_plan_create(w.rows, w.cols, offsets, dtype=w.dtype, schedule=schedule,
                               topology=topology, home_xcd=home_xcd, device=0)
    try:
        bsm.bsm_plan_execute(plan, x, out, trace=trace)
        torch.cuda.synchronize()
        stats = bsm.bsm_plan_describe(plan)
    finally:
        plan.destroy()
    return out, stats


def oracle_full(w, nthreads=16):
    return oracle.softmax(w.x, w.dtype, w.offsets[: w.batch], w.rows, w.cols, nthreads=nthreads)


# ------------------------------------------------------------------------------- backward
def backward_inputs(w, seed=1000, nthreads=16):
    """Seeded inputs of the backward pass for workload w: y = the oracle's softmax of w.x rounded
    to w's dtype (0 outside the slices), dy = workloads.gradient(w). Returns (y, dy) as host
    arrays in w's storage dtype (bf16 as bit patterns)."""
    import workloads

    y64 = oracle.softmax(w.x, w.dtype, w.offsets[: w.batch], w.rows, w.cols, nthreads=nthreads)
    y32 = np.nan_to_num(y64, nan=0.0).astype(np.float32)
    y = workloads._to_bf16_bits(y32) if w.dtype == "bf16" else y32
    return y, workloads.gradient(w, seed)


def _as_f64(a, dtype):
    if dtype == "f32":
        return a.astype(np.float64)
    return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def backward_tolerance(y, dy, dtype, offsets, rows, cols):
    """Per-element bound on |dx - dx_ref| for fp32 arithmetic on the given inputs, derived from
    the kernel's operations: d is a tree sum of C rounded products, so |d - d_ref| <=
    (ceil(log2 C) + 1) u sum_k |y_k dy_k|; dx = y (dy - d) adds two roundings,
    2 u |y| (|dy| + |d|).  u = 2^-24; the bound is doubled for second-order terms."""
    y64, d64 = _as_f64(y, dtype), _as_f64(dy, dtype)
    tol = np.zeros(y64.shape[0])
    u = 2.0 ** -24
    for o, R, C in zip(offsets, rows, cols):
        o, R, C = int(o), int(R), int(C)
        if R == 0 or C == 0:
            continue
        ys = y64[o:o + R * C].reshape(R, C)
        ds = d64[o:o + R * C].reshape(R, C)
        prod = ys * ds
        sabs = np.abs(prod).sum(axis=1, keepdims=True)
        d = prod.sum(axis=1, keepdims=True)
        k = int(np.ceil(np.log2(C))) + 1 if C > 1 else 1
        t = np.abs(ys) * (k * u * sabs + 2 * u * (np.abs(ds) + np.abs(d)))
        tol[o:o + R * C] = 2.0 * t.reshape(-1)
    return tol


def compare_backward(dx_bits, ref, y, dy, dtype, offsets, rows, cols, mask=None):
    """Checks GPU dx against the fp64 oracle within the derived bound (fp32), or 2^-8 relative
    plus twice that bound (bf16: one final rounding). NaN positions must agree."""
    got = bits_to_f64(dx_bits)
    tol = backward_tolerance(y, dy, dtype, offsets, rows, cols)
    if dtype == "bf16":
        tol = 2.0 ** -8 * np.abs(np.nan_to_num(ref)) + 2.0 * tol
    if mask is not None:
        got, ref, tol = got[mask], ref[mask], tol[mask]
    nan_ref = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan_ref), "NaN positions differ"
    err = np.abs(got[~nan_ref] - ref[~nan_ref])
    bad = err > tol[~nan_ref]
    assert not bad.any(), (f"{int(bad.sum())} of {err.size} dx beyond the bound; worst excess "
                           f"{float((err - tol[~nan_ref]).max()):.3e}")
    return float(err.max()) if err.size else 0.0


def run_plan_backward(w, y, dy, schedule="xcd", dx=None, topology=None, trace=None):
    """Backward through bsm_plan_create/execute_backward; y, dy device tensors. Returns
    (dx tensor, plan stats)."""
    n = int(w.offsets[-1]) if len(w.offsets) else 0
    if dx is None:
        dx = sentinel_like(max(n, 1), w.dtype)
    plan = bsm.bsm_plan_create(w.rows, w.cols, w.offsets[: w.batch], dtype=w.dtype,
                               schedule=schedule, topology=topology, device=0)
    try:
        bsm.bsm_plan_execute_backward(plan, y, dy, dx, trace=trace)
        torch.cuda.synchronize()
        stats = bsm.bsm_plan_describe(plan)
    finally:
        plan.destroy()
    return dx, stats
