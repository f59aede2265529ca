"""GPU parity of the fused score product + row softmax (bsm_gemm layout "nt_softmax": P_b = row
softmax of alpha Q_b K_b^T, Section 6's score product followed by Section 2's softmax) against
the fp64 oracle: the paper's size (batch 384, 512 x 512 scores of d = 64) under every schedule,
tails in every dimension (partial row rounds, partial column blocks, a reduction past one
64-deep slice), both output types, k = 0, and bit-identical results across schedules."""

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


def _bound(a, b, batch, m, n, k, alpha, out):
    """Per-element bound on |P - P_ref|. A score's error is at most e = 2 (k + 1) u |alpha|
    sum |q||k| (u = 2^-24: k fp32 additions of exact products and the scaling by alpha); a
    probability p_i = e^(s_i - M) / sum_j e^(s_j - M) then moves by at most |ds_i| + max_j |ds_j|
    relative, and the fp32 exponent (s - M) log2 e adds about |s - M| 2^-24 relative (2^-22
    with margin, plus 16 ulp for the sum, the reciprocal and 2^x). bf16 output adds 2^-8."""
    ref = og.scores_softmax(a, b, batch, m, n, k, alpha).reshape(-1, max(n, 1))
    if k == 0:
        e = np.zeros_like(ref)
        s = np.zeros_like(ref)
    else:
        s = og.batched_gemm(a, b, batch, m, n, k, "nt", alpha).reshape(-1, n)
        e = 2.0 * (k + 1) * 2.0 ** -24 * abs(alpha) * og.abs_product_sums(a, b, batch, m, n, k, "nt").reshape(-1, n)
    rel = 2.0 * e.max(axis=1, keepdims=True) + (np.abs(s - s.max(axis=1, keepdims=True)) + 16.0) * 2.0 ** -22
    tol = ref * rel + 1e-30
    if out == "bf16":
        tol = 2.0 ** -8 * ref + 2.0 * tol
    return ref.reshape(-1), tol.reshape(-1)


def _check(got_bits, a, b, batch, m, n, k, alpha, out):
    ref, tol = _bound(a, b, batch, m, n, k, alpha, out)
    got = bits_to_f64(got_bits)
    err = np.abs(got - ref)
    bad = ~(err <= tol)
    assert not bad.any(), (f"{int(bad.sum())} of {err.size} beyond the bound; worst err "
                           f"{float(np.nanmax(err)):.3e}")
    sums = got.reshape(-1, n).sum(axis=1)
    assert np.all(np.abs(sums - 1.0) <= (n * 2.0 ** -8 if out == "bf16" else 1e-4))


def _run(batch, m, n, k, out, schedule, a_d, b_d, alpha):
    tdt = torch.float32 if out == "f32" else torch.bfloat16
    c = torch.full((batch * m * n,), float("nan"), dtype=tdt, device="cuda")
    p = bsm.bsm_gemm_plan_create(batch, m, n, k, "nt_softmax", out, schedule, device=0)
    bsm.bsm_gemm_execute(p, a_d, b_d, c, alpha)
    torch.cuda.synchronize()
    p.destroy()
    return to_host_bits(c)


@pytest.mark.parametrize("out", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(3, 200, 136, 64), (2, 130, 520, 72), (4, 64, 64, 16),
                                   (1, 257, 1000, 128), (2, 33, 9, 8), (2, 70, 203, 20)],
                         ids=["tails", "k72", "small", "wide", "narrow", "elementwise"])
def test_scores_softmax_tails_all_schedules(shape, out):
    batch, m, n, k = shape
    print(f"[nt_softmax {shape} {out}]", flush=True)
    a, b = _operands(batch, m, n, k, seed=80 + m)
    a_d, b_d = _dev_bf16(a), _dev_bf16(b)
    alpha = 1.0 / np.sqrt(k)
    first = None
    for schedule in SCHEDULES:
        got = _run(batch, m, n, k, out, schedule, a_d, b_d, alpha)
        if first is None:
            first = got
            _check(got, a, b, batch, m, n, k, alpha, out)
        else:
            assert np.array_equal(got, first), f"{schedule} differs from rr"


@pytest.mark.parametrize("out", ["bf16", "f32"])
def test_scores_softmax_paper_size(out):
    """384 x (512 x 64)(64 x 512), alpha = 1/8: every output of BALANCED against the oracle,
    RR and XCD bit for bit against BALANCED."""
    batch, m, n, k = 384, 512, 512, 64
    a, b = _operands(batch, m, n, k, seed=90)
    a_d, b_d = _dev_bf16(a), _dev_bf16(b)
    got = _run(batch, m, n, k, out, "balanced", a_d, b_d, 0.125)
    _check(got, a, b, batch, m, n, k, 0.125, out)
    for schedule in ("rr", "xcd"):
        assert np.array_equal(_run(batch, m, n, k, out, schedule, a_d, b_d, 0.125), got)


def test_scores_softmax_large_logits_and_k0():
    """Logits far from 0 (alpha = 4: scores up to ~100, exponent differences that underflow
    fp32 for most columns) stay within the bound; k = 0 gives 1/n everywhere."""
    batch, m, n, k = 2, 96, 200, 64
    a, b = _operands(batch, m, n, k, seed=91)
    got = _run(batch, m, n, k, "f32", "balanced", _dev_bf16(a), _dev_bf16(b), 4.0)
    _check(got, a, b, batch, m, n, k, 4.0, "f32")
    z = torch.zeros(8, dtype=torch.bfloat16, device="cuda")
    got0 = bits_to_f64(_run(batch, m, n, 0, "f32", "balanced", z, z, 1.0))
    assert np.allclose(got0, 1.0 / n, rtol=2.0 ** -20, atol=0)


@pytest.mark.parametrize("k", [64, 72])
def test_scores_softmax_negative_and_zero_alpha(k):
    """alpha < 0: the largest logit comes from the smallest product; alpha = 0: every logit is 0
    and each row is 1/n. Both operand forms (A in registers for k <= 64, through LDS above) and
    a partial last column block (n = 200)."""
    batch, m, n = 2, 80, 200
    a, b = _operands(batch, m, n, k, seed=93 + k)
    a_d, b_d = _dev_bf16(a), _dev_bf16(b)
    for alpha in (-0.5, 0.0):
        got = _run(batch, m, n, k, "f32", "balanced", a_d, b_d, alpha)
        _check(got, a, b, batch, m, n, k, alpha, "f32")
    assert np.allclose(bits_to_f64(got), 1.0 / n, rtol=2.0 ** -20, atol=0)


def test_scores_softmax_temporal_flag_gives_the_same_bits():
    """BSM_FLAG_TEMPORAL only changes the cache hints of P's stores and Q's loads."""
    batch, m, n, k = 16, 256, 512, 64
    a, b = _operands(batch, m, n, k, seed=95)
    a_d, b_d = _dev_bf16(a), _dev_bf16(b)
    outs = []
    for flags in (0, bsm.BSM_FLAG_TEMPORAL):
        p = bsm.bsm_gemm_plan_create(batch, m, n, k, "nt_softmax", "bf16", "balanced",
                                     topology={"flags": flags}, device=0)
        c = torch.empty(batch * m * n, dtype=torch.bfloat16, device="cuda")
        bsm.bsm_gemm_execute(p, a_d, b_d, c, 0.125)
        torch.cuda.synchronize()
        p.destroy()
        outs.append(to_host_bits(c))
    _check(outs[0], a, b, batch, m, n, k, 0.125, "bf16")
    assert np.array_equal(outs[0], outs[1])


@pytest.mark.parametrize("rising", [True, False])
def test_scores_softmax_running_maximum_moves_every_block(rising):
    """Scores that rise (or fall) along each row: with rising scores the running maximum moves
    up in every 64-column block, so the sum kept so far is rescaled 32 times, down to nothing
    for the first blocks; with falling ones it is set by the first block and every later block
    adds terms far below it. Row i's scores are (i + 1) / 8 * j / 64 (+ noise), up to ~256."""
    batch, m, n, k = 2, 64, 2048, 16
    rng = np.random.default_rng(96)
    q = np.zeros((batch, m, k), np.float32)
    q[:, :, 0] = (np.arange(m, dtype=np.float32) + 1.0) / 8.0
    q[:, :, 1:] = 0.05 * rng.standard_normal((batch, m, k - 1), dtype=np.float32)
    key = np.zeros((batch, n, k), np.float32)
    ramp = np.arange(n, dtype=np.float32) / 64.0
    key[:, :, 0] = ramp if rising else ramp[::-1]
    key[:, :, 1:] = rng.standard_normal((batch, n, k - 1), dtype=np.float32)
    a = workloads._to_bf16_bits(q.reshape(-1))
    b = workloads._to_bf16_bits(key.reshape(-1))
    got = _run(batch, m, n, k, "f32", "balanced", _dev_bf16(a), _dev_bf16(b), 1.0)
    _check(got, a, b, batch, m, n, k, 1.0, "f32")


def test_scores_softmax_one_shot():
    batch, m, n, k = 3, 128, 192, 64
    a, b = _operands(batch, m, n, k, seed=92)
    c = torch.empty(batch * m * n, dtype=torch.bfloat16, device="cuda")
    bsm.bsm_gemm(_dev_bf16(a), _dev_bf16(b), c, batch, m, n, k, "nt_softmax", alpha=0.125)
    torch.cuda.synchronize()
    _check(to_host_bits(c), a, b, batch, m, n, k, 0.125, "bf16")


@pytest.mark.parametrize("out", ["bf16", "f32"])
@pytest.mark.parametrize("shape", [(2, 200, 72, 64), (3, 131, 264, 16), (2, 96, 512, 40),
                                   (1, 65, 392, 8), (2, 64, 128, 64), (1, 1, 72, 8), (5, 1, 512, 64),
                                   (3, 33, 136, 24), (2, 80, 200, 72), (2, 130, 512, 128), (1, 97, 264, 104)],
                         ids=["n72", "n264", "n512k40", "n392k8", "n128", "one_row", "rows_of_one",
                              "m33", "k72", "k128", "k104"])
def test_scores_softmax_one_pass_form(shape, out):
    """Shapes of the one-pass form (k <= 128, 64 < n <= 512, 16-byte rows; past k = 64 the A
    rows stay in LDS and each step takes two 64-deep chunks of B): an odd number of
    128-column steps (72, 264, 392: the pair's second wave has no block in the last step),
    partial blocks, ragged row rounds, batches of a single row (the second wave pair of every
    workgroup has no rows and still meets every barrier). The two-pass form (forced by three
    workgroups per CU) gives results within the same bound."""
    batch, m, n, k = shape
    print(f"[nt_softmax one-pass {shape} {out}]", flush=True)
    a, b = _operands(batch, m, n, k, seed=70 + n)
    a_d, b_d = _dev_bf16(a), _dev_bf16(b)
    alpha = 1.0 / np.sqrt(k)
    first = None
    for schedule in SCHEDULES:
        got = _run(batch, m, n, k, out, schedule, a_d, b_d, alpha)
        if first is None:
            first = got
            _check(got, a, b, batch, m, n, k, alpha, out)
        else:
            assert np.array_equal(got, first), f"{schedule} differs from rr"
    tdt = torch.float32 if out == "f32" else torch.bfloat16
    c = torch.full((batch * m * n,), float("nan"), dtype=tdt, device="cuda")
    p = bsm.bsm_gemm_plan_create(batch, m, n, k, "nt_softmax", out, "balanced",
                                 topology={"wg_per_cu": 3}, device=0)
    bsm.bsm_gemm_execute(p, a_d, b_d, c, alpha)
    torch.cuda.synchronize()
    p.destroy()
    _check(to_host_bits(c), a, b, batch, m, n, k, alpha, out)


def test_scores_softmax_one_pass_random_shapes():
    """Seeded random shapes of the one-pass form (64 < n <= 512 in steps of 8, k a multiple of
    8 up to 128, ragged m, alpha of either sign, both output types) against the oracle, and
    RR against BALANCED bit for bit."""
    rng = np.random.default_rng(2002)
    for case in range(10):
        batch = int(rng.integers(1, 4))
        m = int(rng.integers(1, 230))
        n = 8 * int(rng.integers(9, 65))
        k = 8 * int(rng.integers(1, 17))
        alpha = float(rng.choice([-1.0, 1.0]) * rng.uniform(0.05, 0.5))
        out = "bf16" if case % 2 == 0 else "f32"
        print(f"[nt_softmax one-pass random {case}: {batch} {m} {n} {k} {alpha:.3f} {out}]", flush=True)
        a, b = _operands(batch, m, n, k, seed=3000 + case)
        a_d, b_d = _dev_bf16(a), _dev_bf16(b)
        got = _run(batch, m, n, k, out, "balanced", a_d, b_d, alpha)
        _check(got, a, b, batch, m, n, k, alpha, out)
        assert np.array_equal(_run(batch, m, n, k, out, "rr", a_d, b_d, alpha), got)
