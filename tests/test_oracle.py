"""Pins of the fp64 oracle against what the softmax definition fixes (no GPU).

Each check is chosen so that a plausible slip in the oracle fails at least one:
  * a softmax over columns or over the whole slice  -> hand values on 2x3 / 2x2 slices;
  * a dropped max subtraction                        -> +/-1000 rows, bitwise shift invariance;
  * a wrong row stride or slice offset               -> ragged slices with gaps vs torch per slice;
  * a wrong exp argument sign or a dropped term      -> logistic closed form, powers of two, 1/C;
  * a wrong bf16 decode                              -> bf16 rows vs their decoded fp64 values;
  * threading that mixes slices                      -> 1 vs many threads bitwise.
"""

import math

import numpy as np
import pytest
import torch

import oracle
import workloads
from golden_io import hand_values

pytestmark = pytest.mark.filterwarnings("ignore")


def _soft(x, dtype, R, C):
    return oracle.softmax(np.asarray(x), dtype, [0], [R], [C])


@pytest.mark.parametrize("case", hand_values(), ids=lambda c: c["name"])
def test_hand_values_f64(case):
    y = _soft(np.array(case["x"], np.float64), "f64", case["R"], case["C"])
    exp = np.array(case["y"])
    nan = np.isnan(exp)
    assert np.array_equal(np.isnan(y), nan)
    assert np.allclose(y[~nan], exp[~nan], rtol=0, atol=2e-15)
    # exact zeros stay exact zeros
    assert np.all(y[exp == 0.0] == 0.0)


@pytest.mark.parametrize("case", [c for c in hand_values()
                                  if not any(math.isfinite(v) and v != int(v)
                                             for v in c["x"])],
                         ids=lambda c: c["name"])
def test_hand_values_f32_and_bf16(case):
    """Cases whose inputs are exact in fp32 and bf16 give the same result through every
    input type (the conversion to fp64 is exact)."""
    x64 = np.array(case["x"], np.float64)
    y64 = _soft(x64, "f64", case["R"], case["C"])
    y32 = _soft(x64.astype(np.float32), "f32", case["R"], case["C"])
    bits = (x64.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    ybf = _soft(bits, "bf16", case["R"], case["C"])
    assert np.array_equal(y64, y32, equal_nan=True)
    assert np.array_equal(y64, ybf, equal_nan=True)


def test_logistic_closed_form():
    rng = np.random.default_rng(11)
    ab = (rng.standard_normal((200, 2)) * 6).astype(np.float32)
    y = oracle.softmax(ab.reshape(-1), "f32", [0], [200], [2]).reshape(200, 2)
    for (a, b), (y0, y1) in zip(ab.astype(np.float64), y):
        assert abs(y0 - 1.0 / (1.0 + math.exp(b - a))) <= 2e-16 * 4
        assert abs(y1 - 1.0 / (1.0 + math.exp(a - b))) <= 2e-16 * 4


@pytest.mark.parametrize("C", [1, 2, 3, 7, 64, 100, 512, 1000, 4097])
def test_all_equal_row_is_exactly_one_over_c(C):
    x = np.full(3 * C, -2.75, np.float32)
    y = oracle.softmax(x, "f32", [0], [3], [C])
    assert np.all(y == 1.0 / C)


def test_rows_sum_to_one_c1():
    w = workloads.generate("c1")
    y = oracle.softmax(w.x, w.dtype, w.offsets, w.rows, w.cols).reshape(-1, 64)
    err = np.abs(y.sum(axis=1) - 1.0)
    assert err.max() <= 64 * 2.0 ** -52
    assert np.all(y > 0)


@pytest.mark.parametrize("shift", [1, -1, 37, -512, 4096, -4096])
def test_shift_invariance_bitwise(shift):
    """x holds multiples of 2^-8 in [-16, 16]; x + shift is exact in fp32, and the oracle's
    x_j - max is then exact too, so outputs must agree bit for bit."""
    rng = np.random.default_rng(5)
    x = (rng.integers(-4096, 4097, size=24 * 40) / 256.0).astype(np.float32)
    xs = (x + np.float32(shift)).astype(np.float32)
    assert np.array_equal(xs.astype(np.float64) - shift, x.astype(np.float64))
    y0 = oracle.softmax(x, "f32", [0], [24], [40])
    y1 = oracle.softmax(xs, "f32", [0], [24], [40])
    assert np.array_equal(y0, y1)


def test_monotone_within_row():
    rng = np.random.default_rng(6)
    x = np.sort(rng.standard_normal((16, 33)).astype(np.float32), axis=1)
    y = oracle.softmax(x.reshape(-1), "f32", [0], [16], [33]).reshape(16, 33)
    assert np.all(np.diff(y, axis=1) >= 0)


def test_torch_float64_softmax_c1():
    """Library special case: torch's CPU fp64 softmax over the last dim of each slice."""
    w = workloads.generate("c1")
    y = oracle.softmax(w.x, w.dtype, w.offsets, w.rows, w.cols)
    ref = torch.softmax(torch.from_numpy(w.x.astype(np.float64)).view(-1, 64), dim=-1)
    assert np.max(np.abs(y - ref.numpy().reshape(-1))) <= 1e-15


def test_ragged_slices_with_gaps_match_torch_per_slice():
    rows = [3, 1, 5, 2, 4, 1]
    cols = [7, 13, 1, 9, 16, 3]
    w = workloads.custom(rows, cols, sigma=4.0, seed=3, gap=5, base=11)
    out = np.full(w.x.shape[0], np.nan)
    oracle.softmax(w.x, "f32", w.offsets[:-1], w.rows, w.cols, out=out)
    covered = np.zeros(w.x.shape[0], bool)
    for s, (R, C) in enumerate(zip(rows, cols)):
        o = int(w.offsets[s])
        sl = torch.from_numpy(w.x[o:o + R * C].astype(np.float64)).view(R, C)
        ref = torch.softmax(sl, dim=-1).numpy().reshape(-1)
        assert np.max(np.abs(out[o:o + R * C] - ref)) <= 1e-15
        covered[o:o + R * C] = True
    assert np.all(np.isnan(out[~covered]))  # gaps and the leading base are never written


def test_bf16_decode_matches_fp64_of_the_same_values():
    w = workloads.generate("c3", batch=2)
    dec = (w.x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    yb = oracle.softmax(w.x, "bf16", w.offsets, w.rows, w.cols)
    yd = oracle.softmax(dec, "f64", w.offsets, w.rows, w.cols)
    assert np.array_equal(yb, yd)
    # the masked tail is exactly zero and each row still sums to one
    y = yb.reshape(2, 512, 512)
    for s in range(2):
        L = int(w.mask_len[s])
        if L:
            assert np.all(y[s, :, 512 - L:] == 0.0)
        assert np.max(np.abs(y[s].sum(axis=1) - 1.0)) <= 512 * 2.0 ** -52


def test_bf16_closed_form():
    # 0x3F80 = 1.0, 0x0000 = 0.0, 0xFF80 = -inf, 0xC000 = -2.0
    x = np.array([0x3F80, 0x0000, 0xFF80, 0xC000], np.uint16)
    y = oracle.softmax(x, "bf16", [0], [1], [4])
    S = math.e + 1.0 + math.exp(-2.0)
    assert np.allclose(y, [math.e / S, 1.0 / S, 0.0, math.exp(-2.0) / S], rtol=0, atol=1e-15)
    assert y[2] == 0.0


def test_one_hot_argmax_closed_form():
    B, R, C = 3, 20, 37
    x = np.zeros((B, R, C), np.float32)
    for s in range(B):
        for r in range(R):
            x[s, r, (131 * s + 17 * r) % C] = 30.0
    off = np.arange(B, dtype=np.int64) * R * C
    y = oracle.softmax(x.reshape(-1), "f32", off, [R] * B, [C] * B).reshape(B, R, C)
    hot = math.exp(30.0) / (math.exp(30.0) + C - 1)
    cold = 1.0 / (math.exp(30.0) + C - 1)
    for s in range(B):
        for r in range(R):
            j = (131 * s + 17 * r) % C
            assert int(np.argmax(y[s, r])) == j
            # left-to-right fp64 summation of C terms: error <= C * 2^-53 of the sum
            assert abs(y[s, r, j] - hot) <= C * 2.0 ** -53
            others = np.delete(y[s, r], j)
            assert np.allclose(others, cold, rtol=1e-14, atol=0)


def test_threads_do_not_change_bits():
    w = workloads.generate("c5", batch=24)
    y1 = oracle.softmax(w.x, w.dtype, w.offsets, w.rows, w.cols, nthreads=1)
    y7 = oracle.softmax(w.x, w.dtype, w.offsets, w.rows, w.cols, nthreads=7)
    assert np.array_equal(y1, y7, equal_nan=True)


def test_sampled_rows_equal_full_result():
    w = workloads.generate("c5", batch=10)
    full = oracle.softmax(w.x, w.dtype, w.offsets, w.rows, w.cols)
    firsts, lens = [], []
    for s in range(10):
        for r in (0, int(w.rows[s]) // 2, int(w.rows[s]) - 1):
            firsts.append(int(w.offsets[s]) + r * int(w.cols[s]))
            lens.append(int(w.cols[s]))
    part = oracle.softmax_rows(w.x, w.dtype, firsts, lens)
    pos = 0
    for f, n in zip(firsts, lens):
        assert np.array_equal(part[pos:pos + n], full[f:f + n])
        pos += n


def test_empty_slices_write_nothing():
    x = np.arange(10, dtype=np.float32)
    y = oracle.softmax(x, "f32", [0, 3, 3], [0, 2, 1], [5, 0, 3])
    assert np.all(np.isnan(y[:3])) and np.all(np.isnan(y[6:]))
    assert np.allclose(y[3:6], torch.softmax(torch.arange(3, 6.0, dtype=torch.float64), 0))


def test_bad_arguments_are_rejected():
    x = np.zeros(8, np.float32)
    with pytest.raises(ValueError):
        oracle.softmax(x, "f32", [0], [-1], [4])
    with pytest.raises(ValueError):
        oracle.softmax(x, "f32", [4], [2], [4])  # past the end
    with pytest.raises(TypeError):
        oracle.softmax(x, "bf16", [0], [1], [4])
