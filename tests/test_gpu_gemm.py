"""GPU parity of the batched matrix products (bsm_gemm_*) against the fp64 oracle: Section 6's
two products at their full size (batch 384) under every schedule, both output types, tails in
every dimension, alpha, the empty reduction, and the one-shot entry point."""

import numpy as np
import pytest
import torch

import paper_2002_07062_amd as bsm
import workloads
from gpu_util import bits_to_f64, to_host_bits
from oracle import gemm as og

pytestmark = pytest.mark.gpu

SCHEDULES = ("rr", "balanced", "xcd")


def _operands(batch, m, n, k, seed):
    rng = np.random.default_rng(seed)
    a = workloads._to_bf16_bits(rng.standard_normal(batch * m * k, dtype=np.float32))
    b = workloads._to_bf16_bits(rng.standard_normal(batch * n * k, dtype=np.float32))
    return a, b


def _dev_bf16(x):
    return torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).cuda()


def _check(c_bits, a, b, batch, m, n, k, layout, out, alpha=1.0):
    ref = og.batched_gemm(a, b, batch, m, n, k, layout, alpha)
    # fp32 accumulation of k exact products: |err| <= k u sum |a||b| (u = 2^-24), doubled
    tol = 2.0 * max(k, 1) * 2.0 ** -24 * abs(alpha) * og.abs_product_sums(a, b, batch, m, n, k, layout)
    if out == "bf16":
        tol = 2.0 ** -8 * np.abs(ref) + 2.0 * tol
    got = bits_to_f64(c_bits)
    err = np.abs(got - ref)
    bad = err > tol
    assert not bad.any(), f"{int(bad.sum())} of {err.size} beyond the bound; worst {float(err.max()):.3e}"
    return float(err.max())


def _run(plan_args, a_d, b_d, c, alpha=1.0):
    p = bsm.bsm_gemm_plan_create(*plan_args, device=0)
    bsm.bsm_gemm_execute(p, a_d, b_d, c, alpha)
    torch.cuda.synchronize()
    p.destroy()
    return c


@pytest.mark.parametrize("out", ["f32", "bf16"])
@pytest.mark.parametrize("layout,shape", [("nt", (384, 512, 512, 64)), ("nn", (384, 512, 64, 512))],
                         ids=["scores_QKt", "context_PV"])
def test_paper_products_all_schedules(layout, shape, out):
    batch, m, n, k = shape
    a, b = _operands(batch, m, n, k, seed=70 if layout == "nt" else 71)
    a_d, b_d = _dev_bf16(a), _dev_bf16(b)
    tdt = torch.float32 if out == "f32" else torch.bfloat16
    first = None
    for schedule in SCHEDULES:
        print(f"[gemm {layout} {shape} {out} {schedule}]", flush=True)
        c = torch.full((batch * m * n,), float("nan"), dtype=tdt, device="cuda")
        _run((batch, m, n, k, layout, out, schedule), a_d, b_d, c)
        bits = to_host_bits(c)
        if first is None:
            err = _check(bits, a, b, batch, m, n, k, layout, out)
            print(f"  max abs err {err:.3e}", flush=True)
            first = bits
        else:
            assert np.array_equal(bits, first), schedule


@pytest.mark.parametrize("layout", ["nt", "nn"])
@pytest.mark.parametrize("shape", [(3, 37, 45, 24), (2, 70, 33, 20), (5, 1, 1, 1), (1, 33, 96, 40),
                                   (4, 64, 200, 136), (2, 40, 36, 16)])
@pytest.mark.parametrize("out", ["f32", "bf16"])
def test_tails_in_every_dimension(layout, shape, out):
    batch, m, n, k = shape
    a, b = _operands(batch, m, n, k, seed=72)
    a_d, b_d = _dev_bf16(a), _dev_bf16(b)
    tdt = torch.float32 if out == "f32" else torch.bfloat16
    for schedule in ("rr", "balanced"):
        c = torch.full((batch * m * n + 5,), float("nan"), dtype=tdt, device="cuda")
        _run((batch, m, n, k, layout, out, schedule), a_d, b_d, c, alpha=0.125)
        bits = to_host_bits(c)
        _check(bits[: batch * m * n], a, b, batch, m, n, k, layout, out, alpha=0.125)
        tail = bits_to_f64(bits[batch * m * n:])
        assert np.all(np.isnan(tail)), "written past C"


def test_empty_reduction_stores_zeros_and_noops():
    a_d = torch.zeros(8, dtype=torch.bfloat16, device="cuda")
    c = torch.full((2 * 3 * 4,), 7.0, device="cuda")
    _run((2, 3, 4, 0, "nt", "f32", "balanced"), a_d, a_d, c)
    assert torch.all(c == 0)
    c.fill_(7.0)
    bsm.bsm_gemm(a_d, a_d, c, 0, 3, 4, 5)  # batch 0: nothing
    torch.cuda.synchronize()
    assert torch.all(c == 7.0)


def test_one_shot_equals_plan_and_rejects_overlap():
    batch, m, n, k = 24, 512, 512, 64
    a, b = _operands(batch, m, n, k, seed=73)
    a_d, b_d = _dev_bf16(a), _dev_bf16(b)
    c1 = torch.empty(batch * m * n, device="cuda")
    c2 = torch.empty_like(c1)
    _run((batch, m, n, k, "nt", "f32", "xcd"), a_d, b_d, c1)
    bsm.bsm_gemm(a_d, b_d, c2, batch, m, n, k, "nt", schedule="xcd")
    bsm.bsm_gemm(a_d, b_d, c2, batch, m, n, k, "nt", schedule="xcd")  # cached plan
    torch.cuda.synchronize()
    assert torch.equal(c1.view(torch.int32), c2.view(torch.int32))
    buf = torch.zeros(batch * m * n, device="cuda")
    with pytest.raises(bsm.BsmError) as e:  # A is C's memory
        bsm.bsm_gemm(buf.view(torch.bfloat16), b_d, buf, batch, m, n, k)
    assert e.value.status == bsm.BSM_ERR_ALIAS


@pytest.mark.parametrize("layout", ["nt", "nt_softmax"])
def test_trace_counts_every_output_row(layout):
    """The trace's row counts add up to the output rows (the one-pass score softmax, whose
    wave pairs share rows, counts each row once)."""
    batch, m, n, k = 96, 512, 512, 64
    a, b = _operands(batch, m, n, k, seed=74)
    a_d, b_d = _dev_bf16(a), _dev_bf16(b)
    c = torch.empty(batch * m * n, device="cuda")
    p = bsm.bsm_gemm_plan_create(batch, m, n, k, layout, "f32", "balanced", device=0)
    st = bsm.bsm_plan_describe(p)
    trace = torch.zeros(st["trace_bytes"], dtype=torch.uint8, device="cuda")
    bsm.bsm_gemm_execute(p, a_d, b_d, c, 0.125, trace=trace)
    torch.cuda.synchronize()
    p.destroy()
    rec = trace.cpu().numpy().view(bsm.TRACE_DTYPE)
    assert int(rec["rows"].sum()) == batch * m
    # one XCD per residue of the workgroup index (dispatch may rotate the grid as a whole)
    rot = (rec["xcc_id"].astype(np.int64) - rec["wg"].astype(np.int64)) % 8
    assert len(set(rot.tolist())) == 1


@pytest.mark.parametrize("layout,shape", [("nt", (12, 200, 130, 72)), ("nn", (12, 200, 72, 136))])
def test_occupancy_and_homes_do_not_change_bits(layout, shape):
    """Plans for one, two or three workgroups per CU, and an XCD plan with caller-given homes,
    cut the rows differently; every output bit is the same (a row's result depends only on
    its operands)."""
    batch, m, n, k = shape
    a, b = _operands(batch, m, n, k, seed=75)
    a_d, b_d = _dev_bf16(a), _dev_bf16(b)
    outs = []
    for topo, sched, homes in [(dict(wg_per_cu=1), "balanced", None), (dict(wg_per_cu=2), "rr", None),
                               (dict(wg_per_cu=3), "xcd", None),
                               (None, "xcd", np.arange(batch, dtype=np.int8) % 8 // 3)]:
        print(f"[gemm {layout} {shape} {topo} {sched} homes={homes is not None}]", flush=True)
        p = bsm.bsm_gemm_plan_create(batch, m, n, k, layout, "f32", sched, home_xcd=homes,
                                     topology=topo, device=0)
        c = torch.full((batch * m * n,), float("nan"), device="cuda")
        bsm.bsm_gemm_execute(p, a_d, b_d, c)
        torch.cuda.synchronize()
        p.destroy()
        outs.append(to_host_bits(c))
    _check(outs[0], a, b, batch, m, n, k, layout, "f32")
    for o in outs[1:]:
        assert np.array_equal(o, outs[0])


@pytest.mark.parametrize("layout", ["nt", "nn"])
@pytest.mark.parametrize("which", ["a", "b", "c"])
def test_misaligned_operand_takes_the_elementwise_path(layout, which):
    """An operand 2 bytes (or C 4 bytes) off a 16-byte boundary cannot use 16-byte accesses;
    the element-wise instance gives the same results as the aligned one."""
    batch, m, n, k = 5, 96, 80, 72
    a, b = _operands(batch, m, n, k, seed=76)
    a_buf = torch.zeros(a.size + 8, dtype=torch.bfloat16, device="cuda")
    b_buf = torch.zeros(b.size + 8, dtype=torch.bfloat16, device="cuda")
    c_buf = torch.full((batch * m * n + 8,), float("nan"), device="cuda")
    oa, ob, oc = (1 if which == "a" else 0), (1 if which == "b" else 0), (1 if which == "c" else 0)
    a_d, b_d, c = a_buf[oa: oa + a.size], b_buf[ob: ob + b.size], c_buf[oc: oc + batch * m * n]
    a_d.copy_(_dev_bf16(a))
    b_d.copy_(_dev_bf16(b))
    _run((batch, m, n, k, layout, "f32", "balanced"), a_d, b_d, c)
    got = to_host_bits(c)
    ref_c = torch.empty(batch * m * n, device="cuda")
    _run((batch, m, n, k, layout, "f32", "balanced"), _dev_bf16(a), _dev_bf16(b), ref_c)
    want = to_host_bits(ref_c)
    _check(got, a, b, batch, m, n, k, layout, "f32")
    # same products, same fp32 accumulation order per MFMA: the aligned and element-wise
    # instances differ only in how operands reach LDS
    assert np.array_equal(got, want)
    rest = bits_to_f64(to_host_bits(c_buf))
    assert np.all(np.isnan(rest[:oc])) and np.all(np.isnan(rest[oc + batch * m * n:])), "written outside C"


@pytest.mark.parametrize("layout,shape", [("nt", (16, 256, 512, 64)), ("nn", (16, 256, 64, 512))])
def test_temporal_flag_gives_the_same_bits(layout, shape):
    """BSM_FLAG_TEMPORAL only changes the cache hints of C's stores and A's loads."""
    batch, m, n, k = shape
    a, b = _operands(batch, m, n, k, seed=77)
    a_d, b_d = _dev_bf16(a), _dev_bf16(b)
    outs = []
    for flags in (0, bsm.BSM_FLAG_TEMPORAL):
        p = bsm.bsm_gemm_plan_create(batch, m, n, k, layout, "bf16", "balanced",
                                     topology={"flags": flags}, device=0)
        assert bsm.bsm_plan_describe(p)["flags"] == flags
        c = torch.empty(batch * m * n, dtype=torch.bfloat16, device="cuda")
        bsm.bsm_gemm_execute(p, a_d, b_d, c)
        torch.cuda.synchronize()
        p.destroy()
        outs.append(to_host_bits(c))
    _check(outs[0], a, b, batch, m, n, k, layout, "bf16")
    assert np.array_equal(outs[0], outs[1])
