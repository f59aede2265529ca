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
