"""GPU edge cases: ragged geometry with gaps, unaligned bases, odd row lengths, rows beyond the
register tile, special values, in-place runs, indexing exactness, empty slices, aliasing,
determinism, the per-wave trace and the copy reference. Oracle: the fp64 CPU reference."""

import math

import numpy as np
import pytest
import torch

import oracle
import paper_2002_07062_amd as bsm
import workloads
from gpu_util import (SENTINEL_BF16, SENTINEL_F32, backward_inputs, compare, compare_backward,
                      covered_mask, oracle_full, run_plan, run_plan_backward, sentinel_like,
                      to_device, to_host_bits)

pytestmark = pytest.mark.gpu

SCHEDULES = ("rr", "balanced", "xcd")
ODD_COLS = [1, 2, 3, 4, 5, 7, 8, 15, 16, 17, 31, 33, 63, 64, 65, 100, 127, 128, 129, 255, 256,
            257, 511, 512, 513, 1000, 1023, 1024, 1025, 2047, 2048, 2049]


def _check_ragged(w, schedule, topology=None):
    n = int(w.offsets[-1])
    out, st = run_plan(w, schedule, topology=topology)
    bits = to_host_bits(out)
    ref = oracle.softmax(w.x, w.dtype, w.offsets[: w.batch], w.rows, w.cols)
    mask = covered_mask(w.offsets[: w.batch], w.rows, w.cols, n)
    compare(bits, ref, w.dtype, mask)
    sentinel = SENTINEL_F32 if w.dtype == "f32" else SENTINEL_BF16
    assert np.all(bits[~mask] == sentinel), "a byte outside every slice was written"
    return bits, st


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("schedule", SCHEDULES)
def test_ragged_odd_cols_with_gaps(dtype, schedule):
    rng = np.random.default_rng(7)
    cols = ODD_COLS
    rows = [int(r) for r in rng.integers(1, 40, size=len(cols))]
    w = workloads.custom(rows, cols, dtype=dtype, sigma=3.0, seed=8, gap=3, base=5)
    print(f"[ragged {dtype} {schedule}] {len(cols)} slices", flush=True)
    _check_ragged(w, schedule)


# Rows beyond the register tile, by kernel class: 16-byte aligned rows first (each tile of the
# workgroup-held path: two rows of <= 3 vectors per lane (fp32), 4, 8 or 16 vectors per lane,
# and the two-pass path past 64 values per lane), an unaligned row last (shifted vectors; it
# makes the plan count one more vector per row for its kernel class), so that every earlier
# slice starts 16-byte aligned.
LONG_COLS = {
    ("f32", 4): [2052, 2500, 3072, 4096, 4100, 6000, 8188, 4095],
    ("bf16", 4): [4104, 5000, 6144, 8184, 4200, 8000, 4097],
    ("f32", 5): [8196, 12000, 16380, 9001],
    ("bf16", 5): [8200, 12000, 16376, 9001],
    ("f32", 6): [16392, 20000, 32768, 32772, 70000, 20001],
    ("bf16", 6): [16392, 24000, 32768, 32776, 70000, 20001],
}


@pytest.mark.parametrize("kclass", [4, 5, 6])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_long_rows_workgroup_held_and_two_pass(dtype, kclass):
    """Rows beyond the register tile, held by a 256-thread workgroup (up to 8192 elements in
    kernel class 4, 16384 in class 5) or a 512-thread one (32768, class 6), or, longer, read
    twice; odd row counts (rows are paired across ranges); against the oracle under every
    schedule, with the same bits under all."""
    cols = LONG_COLS[(dtype, kclass)]
    rows = [3, 5, 2, 3, 2, 3, 2, 3][: len(cols)]
    w = workloads.custom(rows, cols, dtype=dtype, sigma=3.0, seed=9, gap=8)
    results = []
    for schedule in SCHEDULES:
        print(f"[long {dtype} class {kclass} {schedule}] cols {cols}", flush=True)
        bits, st = _check_ragged(w, schedule)
        threads = 512 if kclass == 6 else 256
        assert st["kernel_class"] == kclass and st["wg_threads"] == threads and st["per_wave"] == 0
        results.append(bits)
    assert np.array_equal(results[0], results[1]) and np.array_equal(results[0], results[2])


# Aligned rows whose 16-byte vector count n = cols * elem_bytes / 16 is not a power of two
# leave part of their register tile empty (masked lanes hold -inf and store nothing).
PARTIAL_TILE_COLS = {
    "f32": [12, 20, 48, 68, 96, 132, 200, 252, 260, 400, 516, 800, 1020],  # n = 3 ... 255
    "bf16": [24, 40, 136, 200, 504, 520, 1016],                            # n = 3 ... 127
}


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_partial_tile_widths_all_schedules(dtype):
    """Widths with a partly empty register tile, row counts that leave partial wave steps,
    16-byte aligned slices: every schedule matches the oracle and all three give the same
    bits."""
    cols = PARTIAL_TILE_COLS[dtype]
    rng = np.random.default_rng(21)
    rows = [int(r) for r in rng.integers(1, 90, size=len(cols))]
    gap = 4 if dtype == "f32" else 8
    w = workloads.custom(rows, cols, dtype=dtype, sigma=3.0, seed=22, gap=gap)
    assert all(int(o) * (4 if dtype == "f32" else 2) % 16 == 0 for o in w.offsets)
    results = []
    for schedule in SCHEDULES:
        print(f"[partial tile {dtype} {schedule}] cols {cols}", flush=True)
        bits, _ = _check_ragged(w, schedule)
        results.append(bits)
    assert np.array_equal(results[0], results[1]) and np.array_equal(results[0], results[2])


PACKED_COLS = {"f32": [20, 24, 28, 32, 36, 40, 68, 72, 76, 80, 84, 64, 37, 70],
               "bf16": [40, 48, 56, 64, 72, 80, 136, 144, 152, 160, 168, 128, 73, 140]}


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_packed_tile_widths_all_schedules(dtype):
    """Rows of 5-7, 9-10 and 17-21 vectors in a plan of kernel class 0 (every row <= 64
    vectors): packed groups of exactly that many lanes, 64 / n rows side by side per wave, and
    rows of 8 vectors in eight 8-lane groups, with row counts
    that leave partly filled waves and steps; a power-of-two slice and two unaligned ones in the
    same plan. Every schedule matches the oracle and all three give the same bits."""
    cols = PACKED_COLS[dtype]
    rng = np.random.default_rng(23)
    rows = [int(r) for r in rng.integers(1, 120, size=len(cols))]
    w = workloads.custom(rows, cols, dtype=dtype, sigma=3.0, seed=24, gap=4 if dtype == "f32" else 8)
    results = []
    for schedule in SCHEDULES:
        print(f"[packed tile {dtype} {schedule}] cols {cols} rows {rows}", flush=True)
        bits, st = _check_ragged(w, schedule)
        assert st["kernel_class"] == 0
        results.append(bits)
    assert np.array_equal(results[0], results[1]) and np.array_equal(results[0], results[2])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_partial_tile_special_values_stay_in_their_row(dtype):
    """Rows handled side by side in one wave step: a NaN, +inf or fully masked row changes only
    itself."""
    C = 132 if dtype == "f32" else 200  # n = 33 / 25
    R = 9
    rows = np.random.default_rng(23).standard_normal((R, C)).astype(np.float32) * 4
    rows[1, :] = -np.inf
    rows[2, 7] = np.nan
    rows[4, C - 1] = np.inf
    rows[5, 3:] = -np.inf
    rows[7, :] = 0.0
    x = rows.reshape(-1)
    if dtype == "bf16":
        x = workloads._to_bf16_bits(x)
    w = workloads.Workload("partial_tile_special", dtype, x, np.array([0, R * C], np.int64),
                           np.array([R], np.int32), np.array([C], np.int32), True)
    for schedule in SCHEDULES:
        out, _ = run_plan(w, schedule)
        bits = to_host_bits(out)
        compare(bits, oracle.softmax(w.x, dtype, [0], [R], [C]), dtype)
        assert np.all(bits[C:2 * C] == 0)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_offsets_beyond_2_32_elements(dtype):
    """Slices placed past 2^31 and 2^32 elements and straddling both, in buffers of more than
    2^32 elements (17 GB per fp32 buffer): 64-bit indexing end to end. Only the slices and a
    guard band around each are uploaded and read back."""
    rows = [7, 5, 3, 9, 4]
    cols = [300, 1000, 4096, 64, 513]
    offs = [(1 << 31) - 700, (1 << 31) + 12344, (1 << 32) - 6144, (1 << 32) + (1 << 20),
            (1 << 32) + (1 << 21) + 3]
    n = max(o + r * c for o, r, c in zip(offs, rows, cols)) + 4096
    guard = 256
    # compact host copy: the same slices packed back to back, guards in between
    cw = workloads.custom(rows, cols, dtype=dtype, sigma=3.0, seed=51, gap=2 * guard, base=guard)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    x = torch.zeros(n, dtype=tdt, device="cuda")
    out = sentinel_like(1, dtype).expand(n).contiguous()
    xc = to_device(cw.x, dtype)
    for o, co, R, C in zip(offs, cw.offsets[:-1], rows, cols):
        x[o:o + R * C] = xc[int(co):int(co) + R * C]
    ref = oracle.softmax(cw.x, dtype, cw.offsets[:-1], cw.rows, cw.cols)
    sentinel = SENTINEL_F32 if dtype == "f32" else SENTINEL_BF16
    for schedule in SCHEDULES:
        print(f"[big offsets {dtype} {schedule}] n = {n}", flush=True)
        plan = bsm.bsm_plan_create(rows, cols, offs, dtype=dtype, schedule=schedule, device=0)
        bsm.bsm_plan_execute(plan, x, out)
        torch.cuda.synchronize()
        plan.destroy()
        for o, co, R, C in zip(offs, cw.offsets[:-1], rows, cols):
            co = int(co)
            got = to_host_bits(out[o:o + R * C])
            compare(got, ref[co:co + R * C], dtype)
            assert np.all(to_host_bits(out[o - guard:o]) == sentinel)
            assert np.all(to_host_bits(out[o + R * C:o + R * C + guard]) == sentinel)
        out.view(torch.int32 if dtype == "f32" else torch.int16).fill_(
            int(sentinel.view(np.int32 if dtype == "f32" else np.int16)))
    del x, out
    torch.cuda.empty_cache()


@pytest.mark.parametrize("shift", [1, 2, 3])
def test_unaligned_base_pointer(shift):
    """Input and output start a few elements past a 16-byte boundary: the element-wise path."""
    w = workloads.custom([7, 5, 9, 4], [64, 512, 1000, 3000], sigma=2.0, seed=10)
    n = int(w.offsets[-1])
    buf = torch.zeros(n + shift, device="cuda")
    buf[shift:] = to_device(w.x, "f32")
    x = buf[shift:]
    assert x.data_ptr() % 16 != 0
    outb = sentinel_like(n + shift, "f32")
    out = outb[shift:]
    out_t, _ = run_plan(w, "xcd", x=x, out=out)
    ref = oracle.softmax(w.x, "f32", w.offsets[:-1], w.rows, w.cols)
    compare(to_host_bits(out_t), ref, "f32")


# Rows whose start or length is not a whole number of 16-byte vectors (aligned buffers): read
# as the aligned vectors that cover them, outside elements masked, the first and last vectors
# stored element by element.  Contiguous rows then share their boundary vectors.
SHIFTED_COLS = [1, 2, 3, 5, 7, 9, 13, 30, 77, 129, 333, 1001, 2047, 2051, 4097, 8193, 12001]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_shifted_rows_all_schedules_in_place(dtype):
    """Every width and every start phase (odd gaps): against the oracle, bytes outside the
    slices untouched, the same bits under every schedule, in place equal to out of place, and
    the backward pass against its oracle."""
    rng = np.random.default_rng(31)
    rows = [int(r) for r in rng.integers(1, 12, size=len(SHIFTED_COLS))]
    w = workloads.custom(rows, SHIFTED_COLS, dtype=dtype, sigma=3.0, seed=32, gap=1, base=3)
    x = to_device(w.x, dtype)
    results = []
    for schedule in SCHEDULES:
        print(f"[shifted {dtype} {schedule}]", flush=True)
        bits, st = _check_ragged(w, schedule)
        results.append(bits)
    assert np.array_equal(results[0], results[1]) and np.array_equal(results[0], results[2])
    y = x.clone()
    run_plan(w, "balanced", x=y, out=y)
    n = int(w.offsets[-1])
    mask = covered_mask(w.offsets[: w.batch], w.rows, w.cols, n)
    assert np.array_equal(to_host_bits(y)[mask], results[0][mask])
    assert np.array_equal(to_host_bits(y)[~mask], to_host_bits(x)[~mask])
    yb, dyb = backward_inputs(w)
    ref = oracle.softmax_backward(yb, dyb, dtype, w.offsets[: w.batch], w.rows, w.cols, nthreads=16)
    first = None
    for schedule in SCHEDULES:
        dx, _ = run_plan_backward(w, to_device(yb, dtype), to_device(dyb, dtype), schedule)
        bits = to_host_bits(dx)
        compare_backward(bits, ref, yb, dyb, dtype, w.offsets[: w.batch], w.rows, w.cols, mask)
        sentinel = SENTINEL_F32 if dtype == "f32" else SENTINEL_BF16
        assert np.all(bits[:n][~mask] == sentinel), "a byte outside every slice was written"
        first = bits if first is None else first
        assert np.array_equal(bits, first), schedule


def test_in_place_equals_out_of_place():
    w = workloads.generate("c5", batch=40)
    x = to_device(w.x, w.dtype)
    out, _ = run_plan(w, "xcd", x=x)
    y = x.clone()
    run_plan(w, "xcd", x=y, out=y)
    assert torch.equal(y.view(torch.int32), out.view(torch.int32))


def test_repeat_runs_are_bitwise_identical():
    w = workloads.generate("c2", batch=48)
    x = to_device(w.x, w.dtype)
    a, _ = run_plan(w, "balanced", x=x)
    b, _ = run_plan(w, "balanced", x=x)
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))


@pytest.mark.parametrize("C", [37, 64, 128, 512, 1000])
def test_one_hot_argmax_exact(C):
    B, R = 5, 33
    x = np.zeros((B, R, C), np.float32)
    for s in range(B):
        for r in range(R):
            x[s, r, (131 * s + 17 * r) % C] = 30.0
    w = workloads.Workload("onehot", "f32", x.reshape(-1),
                           np.arange(B + 1, dtype=np.int64) * R * C,
                           np.full(B, R, np.int32), np.full(B, C, np.int32), True)
    out, _ = run_plan(w, "xcd")
    y = out.cpu().numpy().reshape(B, R, C)
    for s in range(B):
        for r in range(R):
            assert int(np.argmax(y[s, r])) == (131 * s + 17 * r) % C
    hot = math.exp(30.0) / (math.exp(30.0) + C - 1)
    assert np.max(np.abs(y.max(axis=2) - hot)) <= 2e-6


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_special_values(dtype):
    """Fully masked rows give zeros; a NaN or +inf entry makes its whole row NaN; partially
    masked rows ignore the masked entries."""
    C = 96
    rows = np.random.default_rng(3).standard_normal((6, C)).astype(np.float32)
    rows[0, :] = -np.inf
    rows[1, 10] = np.nan
    rows[2, 50] = np.inf
    rows[3, 40:] = -np.inf
    rows[4, :] = 0.0
    x = rows.reshape(-1)
    if dtype == "bf16":
        x = workloads._to_bf16_bits(x)
    w = workloads.Workload("special", dtype, x, np.array([0, 6 * C], np.int64),
                           np.array([6], np.int32), np.array([C], np.int32), True)
    out, _ = run_plan(w, "rr")
    bits = to_host_bits(out)
    ref = oracle.softmax(w.x, dtype, [0], [6], [C])
    compare(bits, ref, dtype)
    assert np.all(bits[:C] == 0)  # +0 for a fully masked row


def test_empty_slices_and_noops():
    w = workloads.custom([0, 4, 3, 0, 2], [9, 0, 17, 5, 33], sigma=1.0, seed=4, gap=2)
    _check_ragged(w, "balanced")
    x = torch.zeros(16, device="cuda")
    out = torch.full_like(x, 7.0)
    bsm.bsm_softmax(x, out, 4, 4, batch=0)  # batch 0: no-op
    bsm.bsm_softmax(x, out, 0, 4, batch=4)  # empty slices: no-op
    torch.cuda.synchronize()
    assert torch.all(out == 7.0)


def test_partial_alias_is_rejected():
    x = torch.zeros(4 * 64 + 8, device="cuda")
    with pytest.raises(bsm.BsmError) as e:
        bsm.bsm_softmax(x[:256], x[4:260], 4, 64, batch=1)
    assert e.value.status == bsm.BSM_ERR_ALIAS


@pytest.mark.parametrize("schedule", SCHEDULES)
def test_trace_xcd_mapping_and_row_counts(schedule):
    w = workloads.generate("c5", batch=64)
    info = bsm.bsm_device_info(0)
    plan = bsm.bsm_plan_create(w.rows, w.cols, w.offsets[:-1], dtype="f32", schedule=schedule)
    st = bsm.bsm_plan_describe(plan)
    trace = torch.zeros(st["trace_bytes"], dtype=torch.uint8, device="cuda")
    x = to_device(w.x, "f32")
    out = torch.empty_like(x)
    bsm.bsm_plan_execute(plan, x, out, trace=trace)
    torch.cuda.synchronize()
    rec = trace.cpu().numpy().view(bsm.TRACE_DTYPE)
    waves = st["wg_threads"] // 64
    assert len(rec) == st["n_wg"] * waves
    assert np.array_equal(rec["wg"], np.repeat(np.arange(st["n_wg"]), waves))
    assert int(rec["rows"].sum()) == int(w.rows.sum())
    assert np.all(rec["t_end"] >= rec["t_start"])
    print(f"n_xcd={info['n_xcd']} xcc ids seen: {sorted(set(rec['xcc_id'].tolist()))}", flush=True)
    if info["n_xcd"] > 1:
        # dispatch deals consecutive workgroups to consecutive XCDs, round robin: workgroup w
        # runs on XCD (w + r) mod n_xcd for one rotation r per launch (r = 0 in nearly every
        # launch; the XCD schedule plans for w mod n_xcd, results never depend on it)
        rot = (rec["xcc_id"].astype(np.int64) - rec["wg"].astype(np.int64)) % info["n_xcd"]
        assert len(set(rot.tolist())) == 1, sorted(set(rot.tolist()))
    plan.destroy()


def test_copy_kernel():
    for n in (1, 15, 16, 1000, 1 << 20, (1 << 20) + 7):
        src = torch.randint(0, 255, (n,), dtype=torch.uint8, device="cuda")
        dst = torch.zeros_like(src)
        bsm.bsm_copy(src, dst)
        torch.cuda.synchronize()
        assert torch.equal(src, dst)
    a = torch.randn(1 << 20, device="cuda")
    b = torch.zeros((1 << 20) + 1, device="cuda")[1:]  # unaligned destination
    bsm.bsm_copy(a, b, a.numel() * 4)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_device_info():
    d = bsm.bsm_device_info(0)
    print(d, flush=True)
    assert d["n_cu"] > 0 and d["wave_size"] == 64
    assert "gfx950" in d["arch"]


def test_plan_cache_eviction_and_reuse():
    """More distinct geometries than the one-shot cache holds: every call stays correct."""
    bsm.bsm_cache_clear()
    rng = np.random.default_rng(21)
    cases = []
    for i in range(40):
        C = int(rng.integers(8, 700))
        R = int(rng.integers(1, 9))
        B = int(rng.integers(1, 6))
        cases.append((B, R, C))
    for rep in range(2):
        for (B, R, C) in cases:
            w = workloads.custom([R] * B, [C] * B, sigma=2.0, seed=B * 1000 + C)
            x = to_device(w.x, "f32")
            out = sentinel_like(x.numel(), "f32")
            bsm.bsm_softmax(x, out, R, C, batch=B, schedule=SCHEDULES[(B + rep) % 3])
            torch.cuda.synchronize()
            ref = oracle.softmax(w.x, "f32", w.offsets[:-1], w.rows, w.cols)
            compare(to_host_bits(out), ref, "f32")
    bsm.bsm_cache_clear()


def test_two_threads_two_streams():
    """Plans built and run concurrently from two host threads on two streams."""
    import threading

    w = workloads.generate("c5", batch=48)
    x = to_device(w.x, w.dtype)
    ref, _ = run_plan(w, "balanced", x=x)
    results, errors = {}, []

    def work(k):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                out = torch.empty_like(x)
                for _ in range(5):
                    bsm.bsm_softmax(x, out, w.rows, w.cols, slice_offsets=w.offsets[:-1],
                                    schedule="balanced")
            s.synchronize()
            results[k] = out
        except Exception as e:  # reported below
            errors.append(e)

    ts = [threading.Thread(target=work, args=(k,)) for k in range(2)]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    assert not errors, errors
    for k in range(2):
        assert torch.equal(results[k].view(torch.int32), ref.view(torch.int32))
    bsm.bsm_cache_clear()


def test_bf16_one_shot_ragged_all_schedules():
    w = workloads.custom([5, 17, 3, 40], [520, 64, 1000, 8], dtype="bf16", sigma=3.0, seed=12,
                         gap=8)
    x = to_device(w.x, "bf16")
    ref = oracle.softmax(w.x, "bf16", w.offsets[:-1], w.rows, w.cols)
    mask = covered_mask(w.offsets[:-1], w.rows, w.cols, x.numel())
    prev = None
    for sch in SCHEDULES:
        out = sentinel_like(x.numel(), "bf16")
        bsm.bsm_softmax(x, out, w.rows, w.cols, slice_offsets=w.offsets[:-1], schedule=sch)
        torch.cuda.synchronize()
        bits = to_host_bits(out)
        compare(bits, ref, "bf16", mask)
        assert np.all(bits[~mask] == SENTINEL_BF16)
        if prev is not None:
            assert np.array_equal(prev, bits)
        prev = bits
    bsm.bsm_cache_clear()


def test_explicit_stream_and_plan_reuse():
    w = workloads.generate("c4", batch=64)
    x = to_device(w.x, w.dtype)
    plan = bsm.bsm_plan_create(w.rows, w.cols, w.offsets[:-1], dtype="f32", schedule="xcd")
    s = torch.cuda.Stream()
    outs = [torch.empty_like(x) for _ in range(3)]
    with torch.cuda.stream(s):
        for o in outs:
            bsm.bsm_plan_execute(plan, x, o)
    s.synchronize()
    plan.destroy()  # waits on the plan's last use
    ref = oracle.softmax(w.x, "f32", w.offsets[:-1], w.rows, w.cols)
    for o in outs:
        compare(to_host_bits(o), ref, "f32")


@pytest.mark.parametrize("cfg", ["c3", "c5"])
def test_temporal_cache_policy_gives_the_same_bits(cfg):
    """BSM_FLAG_TEMPORAL only changes the cache hints of the row accesses."""
    w = workloads.generate(cfg, batch=32)
    x = to_device(w.x, w.dtype)
    a, _ = run_plan(w, "balanced", x=x)
    b, st = run_plan(w, "balanced", x=x, topology={"flags": bsm.BSM_FLAG_TEMPORAL})
    assert st["flags"] == bsm.BSM_FLAG_TEMPORAL
    view = torch.int16 if w.dtype == "bf16" else torch.int32
    assert torch.equal(a.view(view), b.view(view))


@pytest.mark.parametrize("cfg,batch", [("c2", 64), ("c4", 2048), ("c5", 96)])
def test_bank_layouts_give_the_same_bits(cfg, batch):
    """Interleaved (default) and contiguous virtual banks home the slices on different XCDs;
    the outputs are identical to each other and to BALANCED, and the default homes of a uniform
    batch follow the interleaving (C2: slice s on XCD s mod 8; C4: groups of sixteen)."""
    w = workloads.generate(cfg, batch=batch)
    print(f"[{cfg}] batch {batch}", flush=True)
    x = to_device(w.x, w.dtype)
    a, st_a = run_plan(w, "xcd", x=x)
    b, st_b = run_plan(w, "xcd", x=x, topology={"flags": bsm.BSM_FLAG_CONTIGUOUS_BANKS})
    c, _ = run_plan(w, "balanced", x=x)
    assert st_b["flags"] == bsm.BSM_FLAG_CONTIGUOUS_BANKS and st_a["flags"] == 0
    view = torch.int16 if w.dtype == "bf16" else torch.int32
    assert torch.equal(a.view(view), b.view(view))
    assert torch.equal(a.view(view), c.view(view))
    if cfg != "c5":
        plan = bsm.bsm_plan_create(w.rows, w.cols, w.offsets[: w.batch], dtype=w.dtype,
                                   schedule="xcd", device=0)
        _, _, home, _ = bsm.bsm_plan_export(plan)
        plan.destroy()
        s = np.arange(w.batch)
        group = 1 if cfg == "c2" else 16
        assert home.tolist() == ((s // group) % st_a["n_xcd"]).tolist()


def _run_weighted(w, weights, pad=64):
    """Runs w under the weighted XCD plan into a sentinel-filled output `pad` elements longer
    than the slices' extent, with a per-wave trace; returns (output bits, stats, trace)."""
    n = int(w.offsets[-1])
    x = to_device(w.x, w.dtype)
    out = sentinel_like(n + pad, w.dtype)
    plan = bsm.bsm_plan_create(w.rows, w.cols, w.offsets[: w.batch], dtype=w.dtype,
                               schedule="xcd", device=0, xcd_weight=weights)
    st = bsm.bsm_plan_describe(plan)
    trace = torch.zeros(st["trace_bytes"], dtype=torch.uint8, device="cuda")
    bsm.bsm_plan_execute(plan, x, out, trace=trace)
    torch.cuda.synchronize()
    plan.destroy()
    return to_host_bits(out), st, trace.cpu().numpy().view(bsm.TRACE_DTYPE)


def _check_weighted_against_oracle(w, bits, pad):
    """Element by element against the fp64 oracle inside the slices; the sentinel untouched in
    every element outside them (gaps and the tail past the extent)."""
    n = int(w.offsets[-1])
    mask = np.concatenate([covered_mask(w.offsets[: w.batch], w.rows, w.cols, n),
                           np.zeros(pad, bool)])
    ref = np.concatenate([oracle_full(w), np.zeros(pad)])
    compare(bits, ref, w.dtype, mask)
    sentinel = SENTINEL_F32 if w.dtype == "f32" else SENTINEL_BF16
    assert np.all(bits[~mask] == sentinel), "an element outside the slices was written"


def _rotation(rec):
    rot = set(((rec["xcc_id"].astype(np.int64) - rec["wg"].astype(np.int64)) % 8).tolist())
    assert len(rot) == 1, sorted(rot)
    return rot.pop()


def test_weighted_xcd_plan_same_bits_and_weight_zero_xcd_idle():
    """Weighted load balancing (Section 4.2) moves rows between XCDs but never changes a result:
    the output matches the fp64 oracle element by element and the unweighted plan bit for bit,
    the sentinel survives outside the slices, and an XCD of weight 0 runs no rows (per-wave
    trace)."""
    w = workloads.generate("c5", batch=96)
    ref, _ = run_plan(w, "xcd", x=to_device(w.x, "f32"))
    pad = 64
    bits, st, rec = _run_weighted(w, [1, 1, 1, 1, 1, 1, 1, 0], pad)
    _check_weighted_against_oracle(w, bits, pad)
    n = int(w.offsets[-1])
    assert np.array_equal(bits[:n], to_host_bits(ref)[:n])
    # the workers planned for XCD 7 (w mod 8 == 7) run nothing, and so does the XCD that runs
    # them (dispatch may rotate the whole grid by r XCDs)
    rot = _rotation(rec)
    assert rec["rows"][rec["wg"] % 8 == 7].sum() == 0
    assert rec["rows"][rec["xcc_id"] == (7 + rot) % 8].sum() == 0
    assert rec["rows"].sum() == int(w.rows.sum())
    assert st["xcd_bytes"][7] == 0


def test_weighted_xcd_plan_skewed_weights_uniform_batch():
    """64 slices of 512 x 512 fp32 with skewed weights [4, 1, 1, 1, 1, 1, 1, 0.5]: XCD x is given
    a share of the rows in proportion to its weight (every XCD has the same workgroups; whole
    rows, so within two rows of the exact share), the rows each XCD's waves report match the
    plan's per-XCD bytes, and the output matches the fp64
    oracle element by element with the sentinel intact past the extent."""
    w = workloads.generate("c2", batch=64)
    weights = [4, 1, 1, 1, 1, 1, 1, 0.5]
    pad = 128
    bits, st, rec = _run_weighted(w, weights, pad)
    _check_weighted_against_oracle(w, bits, pad)
    row_bytes = 512 * 4 * 2
    total = int(st["algorithmic_bytes"])
    xb = np.array(st["xcd_bytes"][:8], np.int64)
    assert int(xb.sum()) == total
    share = np.array(weights) / sum(weights) * total
    assert np.all(np.abs(xb - share) <= 2 * row_bytes), (xb.tolist(), share.tolist())
    rot = _rotation(rec)
    for x in range(8):
        rows_x = int(rec["rows"][rec["xcc_id"] == (x + rot) % 8].sum())
        assert rows_x * row_bytes == int(xb[x]), (x, rows_x)


@pytest.mark.parametrize("threads", [64, 256, 512, 1024])
def test_bf16_class3_plans_run_at_most_256_thread_workgroups(threads):
    """bf16 rows of 2049-4096 elements (kernel class 3) run in an instance compiled for
    workgroups of up to 256 threads: a larger request runs 256, a smaller one as asked; every
    size matches the oracle."""
    cols = [2304, 4096, 3000, 2056]
    w = workloads.custom([9, 4, 7, 5], cols, dtype="bf16", sigma=3.0, seed=13, gap=8)
    print(f"[bf16 class 3 asked {threads}]", flush=True)
    bits, st = _check_ragged(w, "balanced", topology=dict(wg_threads=threads))
    assert st["kernel_class"] == 3 and st["wg_threads"] == min(threads, 256)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_long_row_plans_run_256_thread_workgroups(dtype):
    """A plan with rows beyond the register tile runs 256-thread workgroups whatever workgroup
    size the topology asks for (a row's bits depend on it): same bits for 64, 256 and 512, and
    the per-wave trace counts every row once."""
    cols = [5000, 6144, 8192, 7000]
    w = workloads.custom([3, 2, 5, 3], cols, dtype=dtype, sigma=3.0, seed=12, gap=8)
    first = None
    for threads in (64, 256, 512):
        print(f"[long-row workgroups {dtype} asked {threads}]", flush=True)
        n = int(w.offsets[-1])
        x = to_device(w.x, dtype)
        out = sentinel_like(n, dtype)
        plan = bsm.bsm_plan_create(w.rows, w.cols, w.offsets[: w.batch], dtype=dtype,
                                   schedule="balanced", device=0,
                                   topology=dict(wg_threads=threads))
        st = bsm.bsm_plan_describe(plan)
        trace = torch.zeros(st["trace_bytes"], dtype=torch.uint8, device="cuda")
        bsm.bsm_plan_execute(plan, x, out, trace=trace)
        torch.cuda.synchronize()
        plan.destroy()
        assert st["wg_threads"] == 256 and st["per_wave"] == 0
        rec = trace.cpu().numpy().view(bsm.TRACE_DTYPE)
        assert int(rec["rows"].sum()) == int(w.rows.sum())
        bits = to_host_bits(out)
        if first is None:
            first = bits
            mask = covered_mask(w.offsets[: w.batch], w.rows, w.cols, n)
            compare(bits, oracle.softmax(w.x, dtype, w.offsets[: w.batch], w.rows, w.cols),
                    dtype, mask)
        assert np.array_equal(bits, first), threads
