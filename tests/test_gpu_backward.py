"""GPU parity of the softmax backward (dx = y * (dy - sum(dy * y)) per row) against the fp64
oracle, through the C ABI: the five workloads at full size under every schedule, ragged odd
widths with gaps, rows beyond the register tile, in-place runs, special values, aliasing."""

import numpy as np
import pytest
import torch

import oracle
import paper_2002_07062_amd as bsm
import workloads
from gpu_util import (SENTINEL_BF16, SENTINEL_F32, backward_inputs, compare_backward,
                      covered_mask, run_plan_backward, sentinel_like, to_device, to_host_bits)

pytestmark = pytest.mark.gpu

SCHEDULES = ("rr", "balanced", "xcd")


def _check(w, schedule, y, dy, yd=None, dyd=None, topology=None):
    n = int(w.offsets[-1])
    yd = to_device(y, w.dtype) if yd is None else yd
    dyd = to_device(dy, w.dtype) if dyd is None else dyd
    dx, st = run_plan_backward(w, yd, dyd, schedule, topology=topology)
    bits = to_host_bits(dx)
    ref = oracle.softmax_backward(y, dy, w.dtype, w.offsets[: w.batch], w.rows, w.cols,
                                  nthreads=16)
    mask = covered_mask(w.offsets[: w.batch], w.rows, w.cols, n)
    err = compare_backward(bits, ref, y, dy, w.dtype, w.offsets[: w.batch], w.rows, w.cols, mask)
    sentinel = SENTINEL_F32 if w.dtype == "f32" else SENTINEL_BF16
    assert np.all(bits[~mask] == sentinel), "a byte outside every slice was written"
    return bits, st, err


@pytest.mark.parametrize("cfg", ["c1", "c2", "c3", "c4", "c5"])
def test_config_backward_all_schedules_match_oracle(cfg):
    w = workloads.generate(cfg)
    y, dy = backward_inputs(w)
    yd, dyd = to_device(y, w.dtype), to_device(dy, w.dtype)
    print(f"[backward {cfg} {SCHEDULES[0]}]", flush=True)
    first, _, err = _check(w, SCHEDULES[0], y, dy, yd, dyd)
    print(f"  max abs err {err:.3e}", flush=True)
    for schedule in SCHEDULES[1:]:  # the same bits under every schedule
        print(f"[backward {cfg} {schedule}]", flush=True)
        dx, _ = run_plan_backward(w, yd, dyd, schedule)
        assert np.array_equal(to_host_bits(dx), first), schedule


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("schedule", SCHEDULES)
def test_backward_ragged_odd_cols_with_gaps(dtype, schedule):
    cols = [1, 3, 4, 7, 8, 17, 33, 64, 65, 127, 129, 255, 256, 257, 513, 1000, 1025, 2049]
    rng = np.random.default_rng(41)
    rows = [int(r) for r in rng.integers(1, 30, size=len(cols))]
    w = workloads.custom(rows, cols, dtype=dtype, sigma=3.0, seed=42, gap=3, base=5)
    y, dy = backward_inputs(w)
    print(f"[backward ragged {dtype} {schedule}]", flush=True)
    _check(w, schedule, y, dy)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_backward_packed_tile_widths_all_schedules(dtype):
    """Rows of 5-7 vectors (fp32 also 9-10 and 17-21) in packed groups and of 8 vectors in
    8-lane groups (plans of kernel class 0), with row counts that leave partly filled waves, a 16-vector slice and an unaligned
    one in the same plan: every schedule matches the oracle and all three give the same bits."""
    cols = {"f32": [20, 24, 28, 32, 36, 40, 68, 72, 84, 64, 21],
            "bf16": [40, 48, 56, 64, 72, 128, 41]}[dtype]
    rng = np.random.default_rng(43)
    rows = [int(r) for r in rng.integers(1, 200, size=len(cols))]
    w = workloads.custom(rows, cols, dtype=dtype, sigma=3.0, seed=44, gap=4 if dtype == "f32" else 8)
    y, dy = backward_inputs(w)
    results = []
    for schedule in SCHEDULES:
        print(f"[backward packed {dtype} {schedule}] cols {cols} rows {rows}", flush=True)
        bits, st, _ = _check(w, schedule, y, dy)
        assert st["kernel_class"] == 0
        results.append(bits)
    assert np.array_equal(results[0], results[1]) and np.array_equal(results[0], results[2])


# Rows past the backward register tile (256 vectors): 16-byte aligned rows first, then
# unaligned ones (which make the plan count one more vector per row for its kernel class).
# Class 3: one wave per row, staged in LDS or read twice.  Class 4: a workgroup holds y and
# dy, two rows of 4 vectors per lane or up to 32 values per lane and stream.  Class 5: up to
# 64 values.  Class 6: a 512-thread workgroup, up to 64 values per lane; longer rows read twice.
BWD_LONG_COLS = {
    ("f32", 3): [1028, 1500, 2044, 1030],
    ("f32", 4): [2052, 3000, 4096, 6000, 8188, 2050, 5003],
    ("f32", 5): [8196, 16380, 10001],
    ("f32", 6): [16392, 32768, 32772, 40000, 20001],
    ("bf16", 3): [2056, 3000, 4088, 2050],
    ("bf16", 4): [4104, 6000, 8184, 4098, 5003],
    ("bf16", 5): [8200, 16376, 10001],
    ("bf16", 6): [16392, 32768, 32776, 40000, 20001],
}


@pytest.mark.parametrize("kclass", [3, 4, 5, 6])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_backward_long_rows(dtype, kclass):
    """Rows past the backward register tile under every schedule, against the oracle, with the
    same bits under all three."""
    cols = BWD_LONG_COLS[(dtype, kclass)]
    rows = [3, 2, 5, 3, 2, 3, 1][: len(cols)]
    w = workloads.custom(rows, cols, dtype=dtype, sigma=3.0, seed=43, gap=8)
    y, dy = backward_inputs(w)
    first = None
    for schedule in SCHEDULES:
        print(f"[backward long {dtype} class {kclass} {schedule}] cols {cols}", flush=True)
        bits, st, _ = _check(w, schedule, y, dy)
        assert st["kernel_class"] == kclass
        if first is None:
            first = bits
        assert np.array_equal(bits, first), schedule


@pytest.mark.parametrize("schedule", ["rr", "balanced"])
def test_backward_consecutive_workgroup_items(schedule):
    """Many slices of 3 rows of 6000 fp32 (one row at a time per workgroup, so a slice ends on
    the slot set the next one starts with): a workgroup runs several such items back to back
    (RR: slices s, s + 512, ...), against the oracle."""
    w = workloads.custom([3] * 1100, [6000] * 1100, dtype="f32", sigma=3.0, seed=45)
    y, dy = backward_inputs(w)
    print(f"[backward consecutive items {schedule}]", flush=True)
    _, st, _ = _check(w, schedule, y, dy)
    assert st["kernel_class"] == 4 and st["n_wg"] < w.batch


def test_backward_in_place_equals_out_of_place():
    w = workloads.generate("c5", batch=32)
    y, dy = backward_inputs(w)
    yd, dyd = to_device(y, "f32"), to_device(dy, "f32")
    ref, _ = run_plan_backward(w, yd, dyd, "balanced")
    for which in ("dy", "y"):
        a, b = to_device(y, "f32"), to_device(dy, "f32")
        dx = b if which == "dy" else a
        out, _ = run_plan_backward(w, a, b, "balanced", dx=dx)
        assert out.data_ptr() == dx.data_ptr()
        m = torch.from_numpy(covered_mask(w.offsets[: w.batch], w.rows, w.cols,
                                          int(w.offsets[-1]))).cuda()
        assert torch.equal(out.view(torch.int32)[m], ref.view(torch.int32)[m]), which


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_backward_special_values(dtype):
    """A NaN in dy makes its row NaN; a fully masked forward row (y = 0) gives dx = 0; the
    other rows of the same wave step are unaffected."""
    C, R = 96, 8
    rng = np.random.default_rng(44)
    x = rng.standard_normal((R, C)).astype(np.float32) * 2
    x[1, :] = -np.inf
    w0 = workloads.Workload("bwd_special", "f32", x.reshape(-1), np.array([0, R * C], np.int64),
                            np.array([R], np.int32), np.array([C], np.int32), True)
    y64 = oracle.softmax(w0.x, "f32", [0], [R], [C])
    g = rng.standard_normal((R, C)).astype(np.float32)
    g[3, 17] = np.nan
    y32, g32 = y64.astype(np.float32), g.reshape(-1)
    if dtype == "bf16":
        y, dy = workloads._to_bf16_bits(y32), workloads._to_bf16_bits(g32)
    else:
        y, dy = y32, g32
    w = workloads.Workload("bwd_special", dtype, y, w0.offsets, w0.rows, w0.cols, True)
    for schedule in SCHEDULES:
        bits, _, _ = _check(w, schedule, y, dy)
        f = (bits.astype(np.uint32) << (16 if dtype == "bf16" else 0)).view(np.float32)
        assert np.all(f[C:2 * C] == 0.0)  # y = 0 row: dx = 0 (sign of dy - d)
        assert np.all(np.isnan(f[3 * C:4 * C])) and not np.isnan(np.delete(f, np.s_[3 * C:4 * C])).any()


def test_backward_one_shot_equals_plan_and_rejects_partial_alias():
    w = workloads.generate("c5", batch=48)
    y, dy = backward_inputs(w)
    yd, dyd = to_device(y, "f32"), to_device(dy, "f32")
    ref, _ = run_plan_backward(w, yd, dyd, "xcd")
    dx = torch.empty_like(yd)
    bsm.bsm_softmax_backward(yd, dyd, dx, w.rows, w.cols, w.offsets[: w.batch], schedule="xcd")
    torch.cuda.synchronize()
    m = torch.from_numpy(covered_mask(w.offsets[: w.batch], w.rows, w.cols,
                                      int(w.offsets[-1]))).cuda()
    assert torch.equal(dx.view(torch.int32)[m], ref.view(torch.int32)[m])
    buf = torch.zeros(4 * 64 + 8, device="cuda")
    with pytest.raises(bsm.BsmError) as e:
        bsm.bsm_softmax_backward(buf[:256], buf[:256], buf[4:260], 4, 64, batch=1)
    assert e.value.status == bsm.BSM_ERR_ALIAS


def test_backward_uniform_one_shot_bf16_and_noops():
    w = workloads.generate("c3", batch=16)
    y, dy = backward_inputs(w)
    yd, dyd = to_device(y, "bf16"), to_device(dy, "bf16")
    dx = sentinel_like(int(w.offsets[-1]), "bf16")
    bsm.bsm_softmax_backward(yd, dyd, dx, 512, 512, batch=16)
    torch.cuda.synchronize()
    ref = oracle.softmax_backward(y, dy, "bf16", w.offsets[:-1], w.rows, w.cols, nthreads=16)
    compare_backward(to_host_bits(dx), ref, y, dy, "bf16", w.offsets[:-1], w.rows, w.cols)
    z = torch.zeros(16, device="cuda")
    o = torch.full_like(z, 7.0)
    bsm.bsm_softmax_backward(z, z, o, 4, 4, batch=0)
    bsm.bsm_softmax_backward(z, z, o, 0, 4, batch=4)
    torch.cuda.synchronize()
    assert torch.all(o == 7.0)
