"""Pins of the schedule checks in oracle/plan_checks.py (no GPU).

The MINIMAX enumeration and LPT are pinned by textbook instances with known optima; the bank
table by the table printed in Section 4.1 of the paper; the coverage check by tables with
mistakes planted on purpose (in test data, never in the library).
"""

import numpy as np
import pytest

from golden_io import paper_bank_table
from oracle import plan_checks as pc


def test_minimax_textbook_instances():
    # Two cores, {3,3} | {2,2,2} is optimal at 6; LPT reaches 7 = (4/3 - 1/6) * 6.
    assert pc.minimax_bruteforce([3, 3, 2, 2, 2], 2)[0] == 6
    assert pc.lpt_makespan([3, 3, 2, 2, 2], 2) == 7
    # Graham's tight instance for three cores: optimum 9, LPT 11 = (4/3 - 1/9) * 9.
    assert pc.minimax_bruteforce([5, 5, 4, 4, 3, 3, 3], 3)[0] == 9
    assert pc.lpt_makespan([5, 5, 4, 4, 3, 3, 3], 3) == 11
    # One core carries everything; enough cores leave only the biggest patch.
    assert pc.minimax_bruteforce([1, 2, 3, 4], 1)[0] == 10
    assert pc.minimax_bruteforce([1, 2, 3, 4], 4)[0] == 4
    assert pc.minimax_bruteforce([], 3)[0] == 0.0


def test_minimax_assignment_is_consistent():
    costs = [7, 1, 4, 4, 2, 6]
    best, a = pc.minimax_bruteforce(costs, 3)
    load = [0, 0, 0]
    for c, k in zip(costs, a):
        load[k] += c
    assert max(load) == best == 8  # total 24 over 3 cores: 8 is the lower bound and reachable


def test_lpt_within_four_thirds_of_optimum():
    rng = np.random.default_rng(1)
    for _ in range(30):
        n, p = int(rng.integers(1, 8)), int(rng.integers(1, 4))
        costs = list(rng.integers(1, 20, size=n))
        opt = pc.minimax_bruteforce(costs, p)[0]
        assert opt <= pc.lpt_makespan(costs, p) <= (4 / 3) * opt + 1e-9


def test_paper_bank_table():
    banks, rows = paper_bank_table()
    off = [r["offset"] for r in rows]
    R = [r["R"] for r in rows]
    C = [r["C"] for r in rows]
    t = pc.bank_table(off, R, C, banks)
    for s, r in enumerate(rows):
        assert [int(c > 0) for c in t["counts"][s]] == r["flags"], r["name"]
        assert t["overlap"][s] == r["overlap"], r["name"]
    N = len(rows)
    assert t["N"].sum() > N  # with overlaps counted in every bank they touch
    assert t["L"].sum() == N  # after resolving each overlap to one bank
    # the overlapping batch holds 40 elements on Hy and 20 on Hz: largest share wins
    assert t["home"][3] == 1
    assert list(t["home"]) == [2, 0, 1, 1, 3]


def test_bank_table_tie_goes_to_lowest_bank():
    # span [0, 200), two banks [0,100) [100,200); slice 1 covers [80, 120): 20 / 20
    t = pc.bank_table([0, 80, 150], [1, 1, 1], [10, 40, 50], 2)
    assert t["overlap"].tolist() == [0, 1, 0]
    assert t["home"].tolist() == [0, 0, 1]


def test_interleaved_banks_by_hand():
    """Four contiguous slices of 65536, 65536, 98304 and 32768 fp32 elements over two banks with
    a 256 KiB smallest chunk: span 262144, mean extent 65536 = 256 KiB, so the chunk is one mean
    slice and the chunks [0, 65536) [65536, 131072) [131072, 196608) [196608, 262144) go to
    banks 0, 1, 0, 1. Slice 2 holds 65536 elements on bank 0 and 32768 on bank 1 (OVERLAP,
    home 0)."""
    sizes = [65536, 65536, 98304, 32768]
    off = np.concatenate([[0], np.cumsum(sizes)[:-1]])
    assert pc.interleave_chunk(off, [1] * 4, sizes, 2, 4, min_chunk_bytes=256 * 1024) == 65536
    t = pc.bank_table(off, [1] * 4, sizes, 2, layout="interleaved", elem_bytes=4,
                      min_chunk_bytes=256 * 1024)
    assert t["counts"].tolist() == [[65536, 0], [0, 65536], [65536, 32768], [0, 32768]]
    assert t["home"].tolist() == [0, 1, 0, 1]
    assert t["overlap"].tolist() == [0, 0, 1, 0]
    assert t["N"].tolist() == [2, 3] and t["L"].tolist() == [2, 2]


def test_interleave_chunk_rules():
    # 1 MiB fp32 slices: the chunk is one slice; 64 KiB slices: sixteen; bf16 halves the bytes
    assert pc.interleave_chunk([0], [512] * 1, [512], 8, 4) == 0  # one slice: contiguous
    off = np.arange(16) * 262144
    assert pc.interleave_chunk(off, [512] * 16, [512] * 16, 8, 4) == 262144
    off = np.arange(256) * 16384
    assert pc.interleave_chunk(off, [128] * 256, [128] * 256, 8, 4) == 16 * 16384
    # 64 such slices make 4 chunks, fewer than the 8 banks: contiguous
    assert pc.interleave_chunk(off[:64], [128] * 64, [128] * 64, 8, 4) == 0
    # bf16: 32 slices of 32 KiB per chunk, and more than 8 such chunks need more than 256
    assert pc.interleave_chunk(off, [128] * 256, [128] * 256, 8, 2) == 0
    off2 = np.arange(512) * 16384
    assert pc.interleave_chunk(off2, [128] * 512, [128] * 512, 8, 2) == 32 * 16384
    # 8 slices of 64x64 fp32 (C1): 8 chunks of 1 MiB exceed the 128 KiB span -> contiguous
    off = np.arange(8) * 4096
    assert pc.interleave_chunk(off, [64] * 8, [64] * 8, 8, 4) == 0
    t = pc.bank_table(off, [64] * 8, [64] * 8, 8, layout="interleaved")
    assert t["home"].tolist() == list(range(8))


def test_bank_bounds_cover_span_exactly():
    b = pc.bank_bounds(10, 27, 8)
    assert b[0] == 10 and b[-1] == 27
    assert all(b[i] <= b[i + 1] for i in range(8))


# geometry for the coverage pins: slice 0 is 5 x 4 at element 0, slice 1 is 1 x 6 at 30
OFF, ROWS, COLS = [0, 30], [5, 1], [4, 6]


def _table(per_worker):
    """per_worker: lists of (elem_offset, cols, nrows, reps, rep_stride)."""
    ptr = [0]
    items = []
    for its in per_worker:
        for (e, c, n, k, st) in its:
            items.append(dict(elem_offset=e, cols=c, nrows=n, reps=k, rep_stride=st))
        ptr.append(len(items))
    return ptr, items


def test_exactly_once_accepts_valid_tables():
    ptr, items = _table([[(0, 4, 3, 1, 0)], [(12, 4, 2, 1, 0), (30, 6, 1, 1, 0)], []])
    assert pc.check_exactly_once(ptr, items, OFF, ROWS, COLS) == []
    # strided: rows 0, 2, 4 and rows 1, 3 of slice 0
    ptr, items = _table([[(0, 4, 1, 3, 2)], [(4, 4, 1, 2, 2), (30, 6, 1, 1, 0)]])
    assert pc.check_exactly_once(ptr, items, OFF, ROWS, COLS) == []


@pytest.mark.parametrize("tables", [
    [[(0, 4, 3, 1, 0)], [(8, 4, 3, 1, 0), (30, 6, 1, 1, 0)]],    # row 2 of slice 0 twice
    [[(0, 4, 3, 1, 0)], [(16, 4, 1, 1, 0), (30, 6, 1, 1, 0)]],   # row 3 of slice 0 missing
    [[(0, 4, 5, 1, 0)], [(30, 6, 2, 1, 0)]],                     # a row past slice 1
    [[(0, 4, 5, 1, 0)], [(30, 4, 1, 1, 0)]],                     # wrong row length
    [[(0, 4, 1, 3, 2)], [(4, 4, 1, 2, 1), (30, 6, 1, 1, 0)]],    # strided overlap
    [[(0, 4, 5, 1, 0)], [(30, 6, 1, 0, 0)]],                     # zero repetitions
])
def test_exactly_once_catches_planted_mistakes(tables):
    ptr, items = _table(tables)
    assert pc.check_exactly_once(ptr, items, OFF, ROWS, COLS) != []


def test_exactly_once_catches_bad_csr():
    ptr, items = _table([[(0, 4, 5, 1, 0)], [(30, 6, 1, 1, 0)]])
    assert pc.check_exactly_once([0, 2, 1], items, OFF, ROWS, COLS) != []
    assert pc.check_exactly_once([0, 1, 3], items, OFF, ROWS, COLS) != []


def test_worker_loads_and_min_moved():
    ptr, items = _table([[(0, 4, 3, 1, 0)], [(12, 4, 2, 1, 0), (30, 6, 1, 1, 0)]])
    loads = pc.worker_loads(ptr, items, row_cost=lambda c: 10 * c, item_cost=1)
    assert loads.tolist() == [121, 142]
    assert pc.min_moved([10, 2, 6], [6, 6, 6]) == 4
    assert pc.min_moved([6, 6], [6, 6]) == 0


def test_weighted_shares_closed_forms():
    """Equal weights give shares proportional to compute units; weights scale them; a bank of
    weight 0 gets nothing; shares always add up to the total."""
    assert pc.weighted_shares(80, [4, 4, 4, 4], [1, 1, 1, 1]) == [20.0] * 4
    assert pc.weighted_shares(80, [2, 6, 4, 4], [7, 7, 7, 7]) == [10.0, 30.0, 20.0, 20.0]
    assert pc.weighted_shares(60, [4, 4, 4], [1, 2, 3]) == [10.0, 20.0, 30.0]
    assert pc.weighted_shares(30, [4, 4, 4], [1, 0, 2]) == [10.0, 0.0, 20.0]
    s = pc.weighted_shares(1000, [3, 5, 2, 7], [0.3, 1.7, 2.0, 0.9])
    assert abs(sum(s) - 1000) < 1e-9
    # min_moved against weighted targets: only the excess over each target moves
    assert pc.min_moved([60, 0, 0], pc.weighted_shares(60, [4, 4, 4], [1, 2, 3])) == 50.0
