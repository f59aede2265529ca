"""Pins of the fp64 softmax-backward oracle against what the mathematics fixes (no GPU).

The backward oracle returns dx = y * (dy - sum(dy * y)) per row. It is checked against things
other than that formula, chosen so that a plausible slip fails at least one:
  * a dropped y factor, a sign error, d taken over the column or the slice
        -> central differences of the (separately pinned) forward oracle; torch autograd;
  * a wrong row stride or slice offset   -> ragged slices with gaps against torch per slice;
  * d summed over dy alone or y alone    -> hand values (constant dy, one-hot y, signed dy);
  * a wrong bf16 decode                  -> bf16 inputs against their decoded fp64 values;
  * threading that mixes slices          -> 1 vs many threads bitwise.
"""

import numpy as np
import pytest
import torch

import oracle
import workloads
from golden_io import backward_hand_values

pytestmark = pytest.mark.filterwarnings("ignore")


def _bwd(y, dy, dtype, R, C):
    return oracle.softmax_backward(np.asarray(y), np.asarray(dy), dtype, [0], [R], [C])


@pytest.mark.parametrize("case", backward_hand_values(), ids=lambda c: c["name"])
def test_hand_values_f64(case):
    y = np.array(case["y"], np.float64)
    dy = np.array(case["dy"], np.float64)
    got = _bwd(y, dy, "f64", case["R"], case["C"])
    want = np.array(case["dx"], np.float64)
    assert np.array_equal(np.isnan(got), np.isnan(want))
    ok = ~np.isnan(want)
    assert np.max(np.abs(got[ok] - want[ok]), initial=0.0) <= 1e-15


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("case", [c for c in backward_hand_values() if c["dyadic"]],
                         ids=lambda c: c["name"])
def test_hand_values_exact_at_every_dtype(dtype, case):
    y = np.array(case["y"], np.float32)
    dy = np.array(case["dy"], np.float32)
    if dtype == "bf16":
        y, dy = workloads._to_bf16_bits(y), workloads._to_bf16_bits(dy)
    got = _bwd(y, dy, dtype, case["R"], case["C"])
    assert np.array_equal(got, np.array(case["dx"], np.float64))


def _loss(x, dy, R, C):
    """L(x) = sum over rows and columns of dy * softmax(x), through the forward oracle."""
    return float(np.sum(dy * oracle.softmax(x, "f64", [0], [R], [C])))


@pytest.mark.parametrize("R,C", [(1, 1), (2, 2), (3, 5), (2, 17)])
def test_central_differences_of_the_forward_oracle(R, C):
    """dx is the gradient of sum(dy * softmax(x)) with respect to x: central differences of the
    forward oracle (pinned on its own) agree to O(h^2)."""
    rng = np.random.default_rng(100 + C)
    x = rng.standard_normal(R * C) * 2.0
    dy = rng.standard_normal(R * C)
    y = oracle.softmax(x, "f64", [0], [R], [C])
    got = _bwd(y, dy, "f64", R, C)
    h = 1e-5
    num = np.empty(R * C)
    for i in range(R * C):
        xp, xm = x.copy(), x.copy()
        xp[i] += h
        xm[i] -= h
        num[i] = (_loss(xp, dy, R, C) - _loss(xm, dy, R, C)) / (2 * h)
    assert np.max(np.abs(got - num)) <= 1e-8


def test_torch_autograd_float64_on_ragged_slices_with_gaps():
    """Slices of different shapes packed with gaps: each slice's dx equals torch's float64
    autograd gradient of sum(dy * softmax(x, dim=-1)); gaps are never written."""
    rows = [3, 1, 4, 2]
    cols = [5, 9, 1, 16]
    w = workloads.custom(rows, cols, dtype="f32", sigma=2.0, seed=31, gap=3, base=2)
    n = int(w.offsets[-1])
    x = w.x.astype(np.float64)
    y = oracle.softmax(x, "f64", w.offsets[:-1], w.rows, w.cols)
    y = np.where(np.isnan(y), 0.0, y)
    dy = np.random.default_rng(32).standard_normal(n)
    got = oracle.softmax_backward(y, dy, "f64", w.offsets[:-1], w.rows, w.cols)
    covered = np.zeros(n, bool)
    for o, R, C in zip(w.offsets[:-1], rows, cols):
        o = int(o)
        xs = torch.tensor(x[o:o + R * C].reshape(R, C), dtype=torch.float64, requires_grad=True)
        (torch.softmax(xs, dim=-1) * torch.tensor(dy[o:o + R * C].reshape(R, C))).sum().backward()
        assert np.max(np.abs(got[o:o + R * C] - xs.grad.numpy().reshape(-1))) <= 1e-14
        covered[o:o + R * C] = True
    assert np.all(np.isnan(got[~covered]))


def test_two_column_closed_form():
    """y = (p, 1-p): dx_0 = p (1 - p) (dy_0 - dy_1) = -dx_1."""
    rng = np.random.default_rng(33)
    R = 64
    p = rng.uniform(0.0, 1.0, R)
    y = np.stack([p, 1.0 - p], axis=1).reshape(-1)
    dy = rng.standard_normal(2 * R)
    got = _bwd(y, dy, "f64", R, 2).reshape(R, 2)
    d = dy.reshape(R, 2)
    want0 = p * (1.0 - p) * (d[:, 0] - d[:, 1])
    assert np.max(np.abs(got[:, 0] - want0)) <= 1e-15
    assert np.max(np.abs(got[:, 1] + want0)) <= 1e-15


def test_gradient_rows_sum_to_zero_and_ignore_a_constant_shift_of_dy():
    """sum_j dx_j = d (1 - sum_j y_j) = 0 for a softmax row, and adding c to every dy_j of a
    row changes dx by c y (1 - sum y) = 0."""
    R, C = 40, 300
    rng = np.random.default_rng(34)
    x = rng.standard_normal(R * C) * 3.0
    y = oracle.softmax(x, "f64", [0], [R], [C])
    dy = rng.standard_normal(R * C)
    dx = _bwd(y, dy, "f64", R, C)
    # rounding bound: C ulps of the row's magnitudes (sum |dx_j| and |d| sum y_j)
    mag = np.abs(dx).reshape(R, C).sum(axis=1) + np.abs((dy * y).reshape(R, C).sum(axis=1))
    assert np.all(np.abs(dx.reshape(R, C).sum(axis=1)) <= C * 2.0 ** -52 * mag)
    dx2 = _bwd(y, dy + 7.0, "f64", R, C)
    assert np.max(np.abs(dx2 - dx)) <= 1e-14


def test_one_hot_dy_gives_a_jacobian_column():
    """dy = e_i: dx_j = y_j (delta_ij - y_i), the i-th column of diag(y) - y y^T."""
    C = 7
    y = oracle.softmax(np.random.default_rng(35).standard_normal(C), "f64", [0], [1], [C])
    for i in range(C):
        dy = np.zeros(C)
        dy[i] = 1.0
        got = _bwd(y, dy, "f64", 1, C)
        want = y * ((np.arange(C) == i) - y[i])
        assert np.max(np.abs(got - want)) <= 1e-16


def test_bf16_decode_matches_fp64_of_the_same_values():
    rng = np.random.default_rng(36)
    R, C = 6, 24
    yb = workloads._to_bf16_bits(rng.uniform(0, 1, R * C).astype(np.float32))
    db = workloads._to_bf16_bits(rng.standard_normal(R * C).astype(np.float32))
    dec = lambda b: (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)  # noqa: E731
    a = _bwd(yb, db, "bf16", R, C)
    b = _bwd(dec(yb), dec(db), "f64", R, C)
    assert np.array_equal(a, b)


def test_threads_do_not_change_bits():
    w = workloads.generate("c5", batch=24)
    n = int(w.offsets[-1])
    y = np.random.default_rng(37).uniform(0, 1, n).astype(np.float32)
    dy = np.random.default_rng(38).standard_normal(n).astype(np.float32)
    a = oracle.softmax_backward(y, dy, "f32", w.offsets[:-1], w.rows, w.cols, nthreads=1)
    b = oracle.softmax_backward(y, dy, "f32", w.offsets[:-1], w.rows, w.cols, nthreads=7)
    assert np.array_equal(a, b, equal_nan=True)


def test_sampled_rows_equal_full_result():
    w = workloads.generate("c5", batch=6)
    n = int(w.offsets[-1])
    y = np.random.default_rng(39).uniform(0, 1, n).astype(np.float32)
    dy = np.random.default_rng(40).standard_normal(n).astype(np.float32)
    full = oracle.softmax_backward(y, dy, "f32", w.offsets[:-1], w.rows, w.cols)
    firsts, lens = [], []
    for s in range(w.batch):
        for r in (0, int(w.rows[s]) - 1):
            firsts.append(int(w.offsets[s]) + r * int(w.cols[s]))
            lens.append(int(w.cols[s]))
    got = oracle.softmax_backward_rows(y, dy, "f32", firsts, lens)
    want = np.concatenate([full[f:f + c] for f, c in zip(firsts, lens)])
    assert np.array_equal(got, want)


def test_bad_arguments_are_rejected():
    y = np.zeros(8, np.float32)
    with pytest.raises(ValueError):
        oracle.softmax_backward(y, np.zeros(7, np.float32), "f32", [0], [2], [4])
    with pytest.raises(ValueError):
        oracle.softmax_backward(y, y, "f32", [0], [3], [4])
    with pytest.raises(TypeError):
        oracle.softmax_backward(y, y, "f64", [0], [2], [4])
