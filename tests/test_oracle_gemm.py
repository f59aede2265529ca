"""Pins of the fp64 batched-GEMM oracle (no GPU). Chosen so that a plausible slip fails one:
  * the wrong operand transposed, or the layouts swapped -> triple loops on tiny inputs, the
    relation nt(A, B) = nn(A, B^T), identity operands;
  * a wrong batch stride                                  -> per-batch distinct tiny inputs;
  * a wrong bf16 decode                                   -> exact small-integer products;
  * alpha dropped or applied twice                        -> power-of-two alpha exactly.
"""

import itertools

import numpy as np
import pytest
import torch

import workloads
from oracle import gemm


def _bf16(x):
    return workloads._to_bf16_bits(np.asarray(x, np.float32))


@pytest.mark.parametrize("layout", ["nt", "nn"])
def test_triple_loops_on_tiny_inputs(layout):
    """Plain Python loops over small integers (exact in bf16 and in every sum)."""
    rng = np.random.default_rng(60)
    batch, m, n, k = 3, 4, 5, 6
    a = rng.integers(-8, 9, size=batch * m * k)
    b = rng.integers(-8, 9, size=batch * n * k)
    got = gemm.batched_gemm(_bf16(a), _bf16(b), batch, m, n, k, layout)
    want = []
    for t, i, j in itertools.product(range(batch), range(m), range(n)):
        s = 0
        for q in range(k):
            av = a[t * m * k + i * k + q]
            bv = b[t * n * k + j * k + q] if layout == "nt" else b[t * k * n + q * n + j]
            s += int(av) * int(bv)
        want.append(s)
    assert got.tolist() == [float(v) for v in want]


def test_nt_equals_nn_with_b_transposed():
    rng = np.random.default_rng(61)
    batch, m, n, k = 5, 7, 9, 11
    a = rng.standard_normal(batch * m * k)
    b = rng.standard_normal(batch * n * k)
    bt = b.reshape(batch, n, k).transpose(0, 2, 1).reshape(-1)
    nt = gemm.batched_gemm(a, b, batch, m, n, k, "nt", dtype="f64")
    nn = gemm.batched_gemm(a, bt, batch, m, n, k, "nn", dtype="f64")
    assert np.array_equal(nt, nn)


def test_identity_operands():
    rng = np.random.default_rng(62)
    batch, n, k = 2, 6, 6
    eye = np.tile(np.eye(k), (batch, 1, 1)).reshape(-1)
    b = rng.integers(-5, 6, size=batch * n * k).astype(np.float64)
    # I @ B^T = B^T and I @ B = B
    nt = gemm.batched_gemm(eye, b, batch, k, n, k, "nt", dtype="f64").reshape(batch, k, n)
    assert np.array_equal(nt, b.reshape(batch, n, k).transpose(0, 2, 1))
    nn = gemm.batched_gemm(eye, b, batch, k, n, k, "nn", dtype="f64").reshape(batch, k, n)
    assert np.array_equal(nn, b.reshape(batch, k, n))


def test_alpha_power_of_two_is_exact():
    rng = np.random.default_rng(63)
    a = _bf16(rng.integers(-4, 5, size=2 * 3 * 8))
    b = _bf16(rng.integers(-4, 5, size=2 * 5 * 8))
    one = gemm.batched_gemm(a, b, 2, 3, 5, 8, "nt")
    eighth = gemm.batched_gemm(a, b, 2, 3, 5, 8, "nt", alpha=0.125)
    assert np.array_equal(eighth, one / 8)


@pytest.mark.parametrize("shape", [(2, 512, 512, 64, "nt"), (2, 512, 64, 512, "nn")])
def test_paper_shapes_against_torch_float64(shape):
    """Section 6's two products at their real sizes (batch cut to 2) against torch's float64
    batched matmul."""
    batch, m, n, k, layout = shape
    rng = np.random.default_rng(64)
    a = _bf16(rng.standard_normal(batch * m * k))
    b = _bf16(rng.standard_normal(batch * n * k))
    got = gemm.batched_gemm(a, b, batch, m, n, k, layout)
    A = torch.from_numpy(gemm._to_f64(a, "bf16").reshape(batch, m, k))
    if layout == "nt":
        B = torch.from_numpy(gemm._to_f64(b, "bf16").reshape(batch, n, k)).transpose(1, 2).contiguous()
    else:
        B = torch.from_numpy(gemm._to_f64(b, "bf16").reshape(batch, k, n))
    want = torch.bmm(A, B).numpy().reshape(-1)
    assert np.max(np.abs(got - want)) <= 1e-12


def test_abs_product_sums_bound_the_products():
    rng = np.random.default_rng(65)
    a = _bf16(rng.standard_normal(3 * 4 * 16))
    b = _bf16(rng.standard_normal(3 * 5 * 16))
    c = gemm.batched_gemm(a, b, 3, 4, 5, 16, "nt")
    s = gemm.abs_product_sums(a, b, 3, 4, 5, 16, "nt")
    assert np.all(np.abs(c) <= s) and np.all(s > 0)


def test_bad_arguments():
    a = _bf16(np.zeros(12))
    with pytest.raises(ValueError):
        gemm.batched_gemm(a, a, 1, 3, 4, 4, "tn")
    with pytest.raises(ValueError):
        gemm.batched_gemm(a, a, 2, 3, 4, 4, "nt")
    with pytest.raises(TypeError):
        gemm.batched_gemm(np.zeros(12, np.float32), a, 1, 3, 4, 4, "nt")
