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


# bf16 bit patterns of the small integers below, written out by hand (sign, 8-bit exponent with
# bias 127, 7-bit mantissa): an independent check of the decode as well.
_BF16_HAND = {0: 0x0000, 1: 0x3F80, -1: 0xBF80, 2: 0x4000, -2: 0xC000, 3: 0x4040,
              -4: 0xC080, 5: 0x40A0, 6: 0x40C0, 0.5: 0x3F00, 7: 0x40E0, 0.25: 0x3E80,
              -3: 0xC040, 4: 0x4080}


def _hand_bits(vals):
    return np.array([_BF16_HAND[v] for v in vals], np.uint16)


@pytest.mark.parametrize("layout", ["nt", "nn"])
def test_abs_product_sums_hand_values(layout):
    """sum_k |a_ik| |b_kj| written out by hand on mixed-sign integers, two batch indices.

    Batch 0: A = [[1, -2, 3], [-1, 0, 2]], B (one key per row, NT) = [[-4, 5, 6], [2, 1, 0]]:
      S[0][0] = 1*4 + 2*5 + 3*6 = 32     (the signed sum is -4 - 10 + 18 = 4)
      S[0][1] = 1*2 + 2*1 + 3*0 = 4      (signed: 2 - 2 + 0 = 0)
      S[1][0] = 1*4 + 0*5 + 2*6 = 16
      S[1][1] = 1*2 + 0*1 + 2*0 = 2      (signed: -2)
    Batch 1: A = [[0.5, 0, -4], [7, 1, -1]], B = [[2, -3, 0.25], [-1, 4, 1]]:
      S[0][0] = 0.5*2 + 0*3 + 4*0.25 = 2
      S[0][1] = 0.5*1 + 0*4 + 4*1 = 4.5
      S[1][0] = 7*2 + 1*3 + 1*0.25 = 17.25
      S[1][1] = 7*1 + 1*4 + 1*1 = 12
    A product of row sums (sum|a| * sum|b|: 6 * 15 = 90 at [0][0]), a missing absolute value,
    a factor of k or 2, or batch 0's B reused for batch 1 each changes some entry."""
    a = [1, -2, 3, -1, 0, 2, 0.5, 0, -4, 7, 1, -1]
    b_nt = [[[-4, 5, 6], [2, 1, 0]], [[2, -3, 0.25], [-1, 4, 1]]]
    if layout == "nt":
        b = [v for batch in b_nt for row in batch for v in row]
    else:  # NN stores B as k x n: the transpose of the NT rows above
        b = [batch[j][q] for batch in b_nt for q in range(3) for j in range(2)]
    s = gemm.abs_product_sums(_hand_bits(a), _hand_bits(b), 2, 2, 2, 3, layout)
    assert s.tolist() == [32.0, 4.0, 16.0, 2.0, 2.0, 4.5, 17.25, 12.0]
    # the decode of the hand-written patterns, through the product itself
    c = gemm.batched_gemm(_hand_bits(a), _hand_bits(b), 2, 2, 2, 3, layout)
    assert c.tolist() == [4.0, 0.0, 16.0, -2.0, 0.0, -4.5, 10.75, -4.0]


def test_abs_product_sums_one_row_hand_values():
    """m = n = 1, k = 4 over two batch indices: sum|a||b| = 3+3+2+2 = 10 and
    0.5*2 + 0*7 + 4*0.25 + 1*3 = 5 (batch 0's B would give 6.5)."""
    a = [1, -1, 2, -2, 0.5, 0, -4, 1]
    b = [3, 3, -1, 1, 2, 7, 0.25, -3]
    for layout in ("nt", "nn"):  # with n = 1 both layouts store B the same way
        s = gemm.abs_product_sums(_hand_bits(a), _hand_bits(b), 2, 1, 1, 4, layout)
        assert s.tolist() == [10.0, 5.0]


def test_scores_softmax_hand_values():
    """Row softmax of alpha A B^T by hand: A = [[1, 0], [0, 2]] (m = 2, k = 2), B = I (n = 2),
    alpha = ln 3: scores [[ln 3, 0], [0, 2 ln 3]], so the rows are [e^ln3, 1] / (3 + 1) =
    [3/4, 1/4] and [1, 9] / 10 = [1/10, 9/10]."""
    a = _hand_bits([1, 0, 0, 2])
    b = _hand_bits([1, 0, 0, 1])
    p = gemm.scores_softmax(a, b, 1, 2, 2, 2, alpha=float(np.log(3.0)))
    assert np.allclose(p, [0.75, 0.25, 0.1, 0.9], rtol=0, atol=1e-15)


def test_scores_softmax_rows_and_degenerate_cases():
    rng = np.random.default_rng(66)
    batch, m, n, k = 3, 5, 7, 16
    a = _bf16(rng.standard_normal(batch * m * k))
    b = _bf16(rng.standard_normal(batch * n * k))
    p = gemm.scores_softmax(a, b, batch, m, n, k, alpha=0.25).reshape(batch * m, n)
    assert np.all(p > 0) and np.allclose(p.sum(axis=1), 1.0, rtol=0, atol=1e-14)
    # a larger score gives a larger probability (the order of each row is kept)
    s = gemm.batched_gemm(a, b, batch, m, n, k, "nt", 0.25).reshape(batch * m, n)
    assert np.array_equal(np.argsort(s, axis=1, kind="stable"), np.argsort(p, axis=1, kind="stable"))
    # alpha = 0 and k = 0: every score is 0, every probability 1/n
    assert np.allclose(gemm.scores_softmax(a, b, batch, m, n, k, alpha=0.0), 1.0 / n, rtol=0, atol=1e-15)
    z = np.zeros(0, np.uint16)
    assert np.allclose(gemm.scores_softmax(z, z, batch, m, n, 0), 1.0 / n, rtol=0, atol=1e-15)
    # n = 1: the single probability is 1
    assert np.allclose(gemm.scores_softmax(a, b[: batch * k], batch, m, 1, k), 1.0, rtol=0, atol=0)
