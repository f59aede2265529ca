"""bsm_softmax_noalloc, the one-shot softmax for callers that cannot allocate device memory:
its work table lives in the library's static device buffer. Checked through the C ABI against
bsm_softmax (bit for bit) and the fp64 oracle, on two calls in a row on one stream, the second
with a smaller input; with device allocations failing; and with a table too large for the
buffer."""

import numpy as np
import pytest
import torch

import oracle
import paper_2002_07062_amd as bsm
import workloads
from gpu_util import compare, covered_mask, sentinel_like, to_device, to_host_bits

pytestmark = pytest.mark.gpu


def _one_shot_ref(w, x, schedule):
    ref = sentinel_like(x.numel(), w.dtype)
    bsm.bsm_softmax(x, ref, w.rows, w.cols, slice_offsets=w.offsets[: w.batch], schedule=schedule)
    return ref


@pytest.mark.parametrize("schedule", ["balanced", "xcd", "rr"])
def test_noalloc_two_calls_in_a_row_match_bsm_softmax(schedule):
    """Call 1: the 384-slice ragged fp32 workload (64..1024-wide slices; the largest table,
    ~3.4 MiB under BALANCED). Call 2, right after on the same stream with no synchronisation:
    64 slices of 512 x 512 fp32, a smaller table over the first one's. Both equal bsm_softmax
    bit for bit and the fp64 oracle within 2e-6, with the sentinel intact past the extent."""
    big = workloads.generate("c5")
    small = workloads.generate("c2", batch=64)
    xb, xs = to_device(big.x, "f32"), to_device(small.x, "f32")
    pad = 64
    ob = sentinel_like(xb.numel() + pad, "f32")
    os_ = sentinel_like(xs.numel() + pad, "f32")
    print(f"[noalloc {schedule}] c5 then c2[:64]", flush=True)
    bsm.bsm_softmax_noalloc(xb, ob, big.rows, big.cols, slice_offsets=big.offsets[:-1],
                            schedule=schedule)
    bsm.bsm_softmax_noalloc(xs, os_, small.rows, small.cols, slice_offsets=small.offsets[:-1],
                            schedule=schedule)
    torch.cuda.synchronize()
    for w, x, o in ((big, xb, ob), (small, xs, os_)):
        n = int(w.offsets[-1])
        bits = to_host_bits(o)
        ref = to_host_bits(_one_shot_ref(w, x, schedule))
        torch.cuda.synchronize()
        assert np.array_equal(bits[:n], ref[:n])
        assert np.all(bits[n:] == np.uint32(0x7FC0DEAD))
        compare(bits[:n], oracle.softmax(w.x, "f32", w.offsets[:-1], w.rows, w.cols, nthreads=16),
                "f32")
    bsm.bsm_cache_clear()


def test_noalloc_bf16_and_repeated_calls():
    """bf16 masked slices (the 384 x 512 x 512 bf16 workload cut to 32 slices), called three
    times in a row into three outputs: all equal bsm_softmax bit for bit and meet the bf16
    bound against the oracle."""
    w = workloads.generate("c3", batch=32)
    x = to_device(w.x, "bf16")
    outs = [sentinel_like(x.numel(), "bf16") for _ in range(3)]
    for o in outs:
        bsm.bsm_softmax_noalloc(x, o, w.rows, w.cols, slice_offsets=w.offsets[:-1])
    torch.cuda.synchronize()
    ref = to_host_bits(_one_shot_ref(w, x, "balanced"))
    torch.cuda.synchronize()
    want = oracle.softmax(w.x, "bf16", w.offsets[:-1], w.rows, w.cols, nthreads=16)
    mask = covered_mask(w.offsets[:-1], w.rows, w.cols, x.numel())
    for o in outs:
        bits = to_host_bits(o)
        assert np.array_equal(bits, ref)
        compare(bits, want, "bf16", mask)
    bsm.bsm_cache_clear()


def test_noalloc_runs_while_device_allocations_fail(monkeypatch):
    """With the test hook failing every work-table allocation, bsm_plan_create returns
    BSM_ERR_OOM but bsm_softmax_noalloc still runs (it allocates none) and stays correct."""
    w = workloads.custom([5, 3, 8], [96, 1000, 64], sigma=3.0, seed=91, gap=16)
    x = to_device(w.x, "f32")
    out = sentinel_like(x.numel(), "f32")
    monkeypatch.setenv("BSM_TEST_ALLOC_FAIL", "device")
    with pytest.raises(bsm.BsmError) as e:
        bsm.bsm_plan_create(w.rows, w.cols, w.offsets[:-1], dtype="f32", device=0)
    assert e.value.status == bsm.BSM_ERR_OOM
    bsm.bsm_softmax_noalloc(x, out, w.rows, w.cols, slice_offsets=w.offsets[:-1])
    torch.cuda.synchronize()
    monkeypatch.delenv("BSM_TEST_ALLOC_FAIL")
    n = x.numel()
    mask = covered_mask(w.offsets[:-1], w.rows, w.cols, n)
    bits = to_host_bits(out)
    compare(bits, oracle.softmax(w.x, "f32", w.offsets[:-1], w.rows, w.cols), "f32", mask)
    assert np.all(bits[~mask] == np.uint32(0x7FC0DEAD))


def test_noalloc_rejects_a_table_beyond_the_buffer():
    """500000 one-row slices of 8, 16 or 24 elements with random gaps: under RR the table holds
    about one 32-byte item per slice (~13 MiB), beyond the 8 MiB buffer. BSM_ERR_INVALID_ARG
    naming the sizes, and nothing is written."""
    B = 500000
    rng = np.random.default_rng(5)
    cols = (8 * rng.integers(1, 4, B)).astype(np.int32)
    rows = np.ones(B, np.int32)
    offs = np.concatenate([[0], np.cumsum(cols + rng.integers(0, 3, B) * 8)])[:B]
    n = int(offs[-1] + cols[-1])
    x = torch.zeros(n, device="cuda")
    out = sentinel_like(n, "f32")
    with pytest.raises(bsm.BsmError) as e:
        bsm.bsm_softmax_noalloc(x, out, rows, cols, slice_offsets=offs, schedule="rr")
    assert e.value.status == bsm.BSM_ERR_INVALID_ARG
    assert "exceeds" in e.value.message and str(bsm.BSM_NOALLOC_SCRATCH_BYTES) in e.value.message
    torch.cuda.synchronize()
    assert np.all(to_host_bits(out) == np.uint32(0x7FC0DEAD))
