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


def test_bank_bounds_cover_span_exactly():
    b = pc.bank_bounds(10, 27, 8)
    assert b[0] == 10 and b[-1] == 27
    assert all(b[i] <= b[i + 1] for i in range(8))


def _table(pairs_per_wg):
    wg_ptr = [0]
    items = []
    for pairs in pairs_per_wg:
        for (s, r0, n) in pairs:
            items.append(dict(slice=s, row_begin=r0, nrows=n))
        wg_ptr.append(len(items))
    return wg_ptr, items


def test_exactly_once_accepts_a_valid_table():
    wg_ptr, items = _table([[(0, 0, 3)], [(0, 3, 2), (1, 0, 1)], []])
    assert pc.check_exactly_once(wg_ptr, items, [5, 1]) == []


@pytest.mark.parametrize("tables", [
    [[(0, 0, 3)], [(0, 2, 3), (1, 0, 1)]],   # row (0,2) twice
    [[(0, 0, 3)], [(0, 4, 1), (1, 0, 1)]],   # row (0,3) missing
    [[(0, 0, 5)], [(1, 0, 2)]],              # row (1,1) does not exist
    [[(0, 0, 5)], [(2, 0, 1)]],              # slice 2 does not exist
])
def test_exactly_once_catches_planted_mistakes(tables):
    wg_ptr, items = _table(tables)
    assert pc.check_exactly_once(wg_ptr, items, [5, 1]) != []


def test_exactly_once_catches_bad_csr():
    wg_ptr, items = _table([[(0, 0, 5)], [(1, 0, 1)]])
    assert pc.check_exactly_once([0, 2, 1], items, [5, 1]) != []
    assert pc.check_exactly_once([0, 1, 3], items, [5, 1]) != []


def test_wg_loads_and_min_moved():
    wg_ptr, items = _table([[(0, 0, 3)], [(0, 3, 2), (1, 0, 1)]])
    loads = pc.wg_loads(wg_ptr, items, row_cost=lambda s: [10, 100][s], item_cost=1)
    assert loads.tolist() == [31, 122]
    assert pc.min_moved([10, 2, 6], [6, 6, 6]) == 4
    assert pc.min_moved([6, 6], [6, 6]) == 0
