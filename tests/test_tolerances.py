"""Hand-derived values of the GPU parity bounds (no GPU).

The backward parity bound (gpu_util.backward_tolerance) is derived from the kernel's operations:
per element, 2 |y_j| (k u sum_i |y_i dy_i| + 2 u (|dy_j| + |d|)), d = sum_i y_i dy_i,
k = ceil(log2 C) + 1 (1 for C = 1), u = 2^-24. The cases below are worked out by hand from that
formula on dyadic values, so the sums are exact; a factor of 2 too many or too few, the absolute
sum replaced by |d| or by sum|y| * sum|dy|, the wrong k, or a row stride or offset slip changes
some entry."""

import numpy as np

from gpu_util import backward_tolerance

U = 2.0 ** -24


def test_backward_tolerance_one_row_of_three():
    """y = [1/2, 1/4, 1/4], dy = [1, -2, 4]: products 1/2, -1/2, 1, sum|.| = 2, d = 1; C = 3 so
    k = 2 + 1 = 3, k u sum|.| = 6u.
      j = 0: 2 * 1/2 * (6u + 2u (1 + 1)) = 10u
      j = 1: 2 * 1/4 * (6u + 2u (2 + 1)) = 6u
      j = 2: 2 * 1/4 * (6u + 2u (4 + 1)) = 8u"""
    y = np.array([0.5, 0.25, 0.25], np.float32)
    dy = np.array([1, -2, 4], np.float32)
    tol = backward_tolerance(y, dy, "f32", [0], [1], [3])
    assert tol.tolist() == [10 * U, 6 * U, 8 * U]


def test_backward_tolerance_two_rows_of_four_with_offset_and_gap():
    """One 2 x 4 slice at element 0, a gap of 2, then the 1 x 3 row above at element 10.
    Row 0: y = [1/8, 1/8, 1/4, 1/2], dy = [8, -8, 2, -1]: products 1, -1, 1/2, -1/2, sum|.| = 3,
    d = 0; C = 4 so k = 3, k u sum|.| = 9u:
      j = 0, 1: 2 * 1/8 * (9u + 16u) = 6.25u;  j = 2: 2 * 1/4 * (9u + 4u) = 6.5u;
      j = 3: 2 * 1/2 * (9u + 2u) = 11u.
    Row 1: y = [1, 0, 0, 0], dy = [3, 5, -7, 9]: sum|.| = 3, d = 3:
      j = 0: 2 * 1 * (9u + 2u (3 + 3)) = 42u; the rest 0 (y = 0).
    The gap gets 0."""
    y = np.array([0.125, 0.125, 0.25, 0.5, 1, 0, 0, 0, 7, 7, 0.5, 0.25, 0.25], np.float32)
    dy = np.array([8, -8, 2, -1, 3, 5, -7, 9, 7, 7, 1, -2, 4], np.float32)
    tol = backward_tolerance(y, dy, "f32", [0, 10], [2, 1], [4, 3])
    want = [6.25, 6.25, 6.5, 11, 42, 0, 0, 0, 0, 0, 10, 6, 8]
    assert tol.tolist() == [v * U for v in want]


def test_backward_tolerance_bf16_inputs_decode():
    """The same 1 x 3 row given as bf16 bit patterns (1/2 = 0x3F00, 1/4 = 0x3E80, 1 = 0x3F80,
    -2 = 0xC000, 4 = 0x4080) gives the same bound; a single column (C = 1, k = 1): y = [1],
    dy = [-3]: 2 * (u * 3 + 2u (3 + 3)) = 30u."""
    y = np.array([0x3F00, 0x3E80, 0x3E80], np.uint16)
    dy = np.array([0x3F80, 0xC000, 0x4080], np.uint16)
    assert backward_tolerance(y, dy, "bf16", [0], [1], [3]).tolist() == [10 * U, 6 * U, 8 * U]
    one = backward_tolerance(np.array([1], np.float32), np.array([-3], np.float32), "f32",
                             [0], [1], [1])
    assert one.tolist() == [30 * U]


def test_bf16_rne_bits_hand_values():
    """Round-to-nearest-even to bf16 on hand-chosen values: exact bf16 values stay; 1 + 2^-8
    (the midpoint between 1 and 1 + 2^-7) goes to the even 1.0 = 0x3F80; 1 + 3 * 2^-8 (the
    midpoint between 1 + 2^-7 and 1 + 2^-6) goes to the even 1 + 2^-6 = 0x3F82; just above a
    midpoint rounds up, just below rounds down; 0 gives +0; 1/3 = 0x3EAB (0.333984375 is
    nearer than 0.33203125)."""
    from gpu_util import bf16_rne_bits, count_non_rne

    v = np.array([1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, 1 + 2 ** -8 + 2 ** -30, 1 + 2 ** -8 - 2 ** -30,
                  0.0, 1 / 3, 0.5, 2 ** -20])
    want = [0x3F80, 0x3F80, 0x3F82, 0x3F81, 0x3F80, 0x0000, 0x3EAB, 0x3F00, 0x3580]
    assert bf16_rne_bits(v).tolist() == want
    bits = np.array(want, np.uint16)
    bits[2] = 0x3F81  # one output rounded the other way
    assert count_non_rne(bits, v) == (1, len(v))
