"""Plain checks of slice-to-workgroup schedules (the paper's Sections 3 to 5).

TEST INFRASTRUCTURE ONLY. Everything here is brute force or a direct definition, written for
clarity rather than speed, and shares no code with the library's host planner:

* exactly-once coverage of every (slice, row) by a work table (the mapping table of
  Section 5 must schedule every patch, and no patch twice);
* the batch-to-bank table of Section 4.1, computed by counting the elements of each slice that
  fall in each bank (OVERLAP flag, the counts N_x with overlaps, the max-proportion home with
  ties to the lowest bank, the counts L_x after resolution);
* the MINIMAX objective of Section 4.2 (min over partitions of the patches of the max summed
  execution time per core), solved by enumerating every assignment for tiny instances;
* longest-processing-time-first list scheduling, a textbook 4/3-approximation of it;
* the least load that any rebalancing must move: the sum of the excesses over the targets.
"""

from __future__ import annotations

import itertools

import numpy as np


# ----------------------------------------------------------------------------- work tables

def table_rows(wg_ptr, items):
    """Expand a CSR work table into (wg, slice, row) triples, one per scheduled row.

    `items` is a structured array or a sequence of dicts with fields slice, row_begin, nrows.
    """
    out = []
    n_wg = len(wg_ptr) - 1
    for w in range(n_wg):
        for i in range(int(wg_ptr[w]), int(wg_ptr[w + 1])):
            it = items[i]
            s, r0, n = int(it["slice"]), int(it["row_begin"]), int(it["nrows"])
            for r in range(r0, r0 + n):
                out.append((w, s, r))
    return out


def check_exactly_once(wg_ptr, items, rows):
    """Return a list of problems (empty when every row of every slice is scheduled exactly
    once and nothing else is)."""
    problems = []
    if int(wg_ptr[0]) != 0:
        problems.append("wg_ptr[0] != 0")
    if any(int(wg_ptr[w + 1]) < int(wg_ptr[w]) for w in range(len(wg_ptr) - 1)):
        problems.append("wg_ptr not monotone")
    if int(wg_ptr[-1]) != len(items):
        problems.append(f"wg_ptr[-1]={int(wg_ptr[-1])} but {len(items)} items")
    if problems:
        return problems
    seen = {}
    for w, s, r in table_rows(wg_ptr, items):
        if not 0 <= s < len(rows) or not 0 <= r < int(rows[s]):
            problems.append(f"row ({s},{r}) does not exist (wg {w})")
            continue
        seen[(s, r)] = seen.get((s, r), 0) + 1
    for (s, r), k in seen.items():
        if k != 1:
            problems.append(f"row ({s},{r}) scheduled {k} times")
    expected = int(sum(int(R) for R in rows))
    if len(seen) != expected:
        problems.append(f"{len(seen)} distinct rows scheduled, {expected} exist")
    return problems


def wg_loads(wg_ptr, items, row_cost, item_cost=0.0):
    """Cost per workgroup: item_cost per item plus row_cost(slice) per row."""
    n_wg = len(wg_ptr) - 1
    loads = np.zeros(n_wg, dtype=np.float64)
    for w in range(n_wg):
        for i in range(int(wg_ptr[w]), int(wg_ptr[w + 1])):
            it = items[i]
            loads[w] += item_cost + int(it["nrows"]) * row_cost(int(it["slice"]))
    return loads


# ----------------------------------------------------------------------- bank table (4.1)

def bank_bounds(lo: int, hi: int, n_banks: int):
    """n_banks equal contiguous element ranges over [lo, hi): bank b = [bound[b], bound[b+1])
    with bound[b] = lo + floor(b * (hi - lo) / n_banks)."""
    span = hi - lo
    return [lo + (b * span) // n_banks for b in range(n_banks + 1)]


def bank_table(offsets, rows, cols, n_banks: int):
    """Batch-to-bank table by counting, element by element, which bank holds each element.

    Banks are n_banks equal contiguous ranges over the elements spanned by the non-empty
    slices. Returns dict with per-slice `counts` [B, n_banks], `overlap` [B] (0/1), `home` [B]
    (bank holding the largest share; ties go to the lowest bank; -1 for an empty slice),
    `N` [n_banks] (slices touching each bank, overlaps counted in every bank they touch) and
    `L` [n_banks] (slices homed on each bank)."""
    B = len(rows)
    sizes = [int(rows[s]) * int(cols[s]) for s in range(B)]
    live = [s for s in range(B) if sizes[s] > 0]
    counts = np.zeros((B, n_banks), dtype=np.int64)
    home = np.full(B, -1, dtype=np.int64)
    overlap = np.zeros(B, dtype=np.int64)
    if not live:
        return dict(counts=counts, overlap=overlap, home=home,
                    N=np.zeros(n_banks, np.int64), L=np.zeros(n_banks, np.int64))
    lo = min(int(offsets[s]) for s in live)
    hi = max(int(offsets[s]) + sizes[s] for s in live)
    bound = bank_bounds(lo, hi, n_banks)
    for s in live:
        for e in range(int(offsets[s]), int(offsets[s]) + sizes[s]):
            b = 0
            while not (bound[b] <= e < bound[b + 1]):
                b += 1
            counts[s, b] += 1
        nz = [b for b in range(n_banks) if counts[s, b] > 0]
        overlap[s] = 1 if len(nz) > 1 else 0
        best = max(counts[s])
        home[s] = min(b for b in range(n_banks) if counts[s, b] == best)
    N = np.array([sum(1 for s in live if counts[s, b] > 0) for b in range(n_banks)])
    L = np.array([sum(1 for s in live if home[s] == b) for b in range(n_banks)])
    return dict(counts=counts, overlap=overlap, home=home, N=N, L=L)


# ---------------------------------------------------------------------------- MINIMAX (4.2)

def minimax_bruteforce(costs, n_cores: int):
    """min over all assignments of whole patches to cores of the max per-core summed cost.
    Enumerates n_cores ** len(costs) assignments: tiny instances only."""
    costs = list(costs)
    if len(costs) == 0:
        return 0.0, ()
    if n_cores ** len(costs) > 2_000_000:
        raise ValueError("instance too large for enumeration")
    best, best_a = None, None
    for a in itertools.product(range(n_cores), repeat=len(costs)):
        load = [0.0] * n_cores
        for c, k in zip(costs, a):
            load[k] += c
        m = max(load)
        if best is None or m < best:
            best, best_a = m, a
    return best, best_a


def lpt_makespan(costs, n_cores: int):
    """Longest processing time first: sort descending, give each patch to the least loaded
    core (lowest index on ties)."""
    load = [0.0] * n_cores
    for c in sorted(costs, reverse=True):
        k = min(range(n_cores), key=lambda i: (load[i], i))
        load[k] += c
    return max(load) if load else 0.0


def min_moved(loads, targets):
    """Least total load any rebalancing must take off the banks: sum of excess over target."""
    return float(sum(max(0.0, float(l) - float(t)) for l, t in zip(loads, targets)))
