"""Plain checks of slice-to-workgroup schedules (the paper's Sections 3 to 5).

TEST INFRASTRUCTURE ONLY. Everything here is brute force or a direct definition, written for
clarity rather than speed, and shares no code with the library's host planner:

* exactly-once coverage of every row of every slice by a work table (the mapping table of
  Section 5 must schedule every patch, and no patch twice), with the slice's row length;
* the batch-to-bank table of Section 4.1, computed by counting the elements of each slice that
  fall in each bank, for contiguous or interleaved virtual banks (OVERLAP flag, the counts N_x
  with overlaps, the max-proportion home with ties to the lowest bank, the counts L_x after
  resolution);
* the MINIMAX objective of Section 4.2 (min over partitions of the patches of the max summed
  execution time per core), solved by enumerating every assignment for tiny instances;
* longest-processing-time-first list scheduling, a textbook 4/3-approximation of it;
* the least load that any rebalancing must move: the sum of the excesses over the targets.
"""

from __future__ import annotations

import itertools

import numpy as np


# ----------------------------------------------------------------------------- work tables
#
# A work table is a CSR row pointer over workers plus items; item i covers `reps` ranges of
# `nrows` rows of row length `cols`, range k starting at element
# elem_offset + k * rep_stride * cols (the library's documented table format).


def slice_row_starts(offsets, rows, cols):
    """Every row of every slice: arrays (start element, slice, row, cols), in slice order."""
    starts, sl, rr, cc = [], [], [], []
    for s in range(len(rows)):
        R, C = int(rows[s]), int(cols[s])
        if R == 0 or C == 0:
            continue
        r = np.arange(R, dtype=np.int64)
        starts.append(int(offsets[s]) + r * C)
        sl.append(np.full(R, s, np.int64))
        rr.append(r)
        cc.append(np.full(R, C, np.int64))
    if not starts:
        z = np.zeros(0, np.int64)
        return z, z, z, z
    return (np.concatenate(starts), np.concatenate(sl), np.concatenate(rr), np.concatenate(cc))


def table_row_starts(worker_ptr, items):
    """Every row a table schedules: arrays (worker, start element, cols)."""
    ws, st, cc = [], [], []
    for v in range(len(worker_ptr) - 1):
        for i in range(int(worker_ptr[v]), int(worker_ptr[v + 1])):
            it = items[i]
            e0, C = int(it["elem_offset"]), int(it["cols"])
            n, reps, stride = int(it["nrows"]), int(it["reps"]), int(it["rep_stride"])
            for k in range(reps):
                first = e0 + k * stride * C
                st.append(first + np.arange(n, dtype=np.int64) * C)
                ws.append(np.full(n, v, np.int64))
                cc.append(np.full(n, C, np.int64))
    if not st:
        z = np.zeros(0, np.int64)
        return z, z, z
    return np.concatenate(ws), np.concatenate(st), np.concatenate(cc)


def check_exactly_once(worker_ptr, items, offsets, rows, cols):
    """Return a list of problems (empty when every row of every slice is scheduled exactly
    once, with its slice's row length, and nothing else is)."""
    problems = []
    if int(worker_ptr[0]) != 0:
        problems.append("worker_ptr[0] != 0")
    if any(int(worker_ptr[w + 1]) < int(worker_ptr[w]) for w in range(len(worker_ptr) - 1)):
        problems.append("worker_ptr not monotone")
    if int(worker_ptr[-1]) != len(items):
        problems.append(f"worker_ptr[-1]={int(worker_ptr[-1])} but {len(items)} items")
    for i in range(len(items)):
        if int(items[i]["reps"]) < 1 or int(items[i]["nrows"]) < 1:
            problems.append(f"item {i} has reps {int(items[i]['reps'])}, nrows {int(items[i]['nrows'])}")
    if problems:
        return problems
    want, _, _, want_c = slice_row_starts(offsets, rows, cols)
    _, got, got_c = table_row_starts(worker_ptr, items)
    order_w, order_g = np.argsort(want, kind="stable"), np.argsort(got, kind="stable")
    if len(got) != len(want):
        problems.append(f"{len(got)} rows scheduled, {len(want)} exist")
        return problems
    if not np.array_equal(want[order_w], got[order_g]):
        dup = np.unique(got[order_g][1:][np.diff(got[order_g]) == 0])
        problems.append(f"scheduled row starts differ from the slices' rows "
                        f"(duplicates: {dup[:5].tolist()})")
        return problems
    if not np.array_equal(want_c[order_w], got_c[order_g]):
        problems.append("a row is scheduled with the wrong row length")
    return problems


def worker_loads(worker_ptr, items, row_cost, item_cost=0.0):
    """Cost per worker: item_cost per item plus row_cost(cols) per row."""
    n = len(worker_ptr) - 1
    loads = np.zeros(n, dtype=np.float64)
    for v in range(n):
        for i in range(int(worker_ptr[v]), int(worker_ptr[v + 1])):
            it = items[i]
            nr = int(it["nrows"]) * int(it["reps"])
            loads[v] += item_cost + nr * row_cost(int(it["cols"]))
    return loads


# ----------------------------------------------------------------------- bank table (4.1)

def bank_bounds(lo: int, hi: int, n_banks: int):
    """n_banks equal contiguous element ranges over [lo, hi): bank b = [bound[b], bound[b+1])
    with bound[b] = lo + floor(b * (hi - lo) / n_banks)."""
    span = hi - lo
    return [lo + (b * span) // n_banks for b in range(n_banks + 1)]


def interleave_chunk(offsets, rows, cols, n_banks: int, elem_bytes: int,
                     min_chunk_bytes: int = 1024 * 1024) -> int:
    """Chunk (elements) of the interleaved virtual banks: the span [lo, hi) of the non-empty
    slices divided by their number (floor, at least 1) is the mean slice extent m; the chunk is
    the smallest multiple of m holding at least min_chunk_bytes. Returns 0 (contiguous banks)
    when n_banks chunks cover the span or there is no non-empty slice."""
    sizes = [int(rows[s]) * int(cols[s]) for s in range(len(rows))]
    live = [s for s in range(len(rows)) if sizes[s] > 0]
    if not live:
        return 0
    lo = min(int(offsets[s]) for s in live)
    hi = max(int(offsets[s]) + sizes[s] for s in live)
    m = max(1, (hi - lo) // len(live))
    k = 1
    while k * m * elem_bytes < min_chunk_bytes:
        k += 1
    chunk = k * m
    return 0 if chunk * n_banks >= hi - lo else chunk


def bank_table(offsets, rows, cols, n_banks: int, layout: str = "contiguous",
               elem_bytes: int = 4, min_chunk_bytes: int = 1024 * 1024):
    """Batch-to-bank table by counting, element by element, which bank holds each element.

    The banks partition the elements spanned by the non-empty slices, [lo, hi). layout
    "contiguous": n_banks equal contiguous ranges. layout "interleaved": element e lies in bank
    floor((e - lo) / chunk) mod n_banks, chunk = interleave_chunk(...), falling back to the
    contiguous ranges where that is 0. Returns dict with per-slice `counts` [B, n_banks],
    `overlap` [B] (0/1), `home` [B] (bank holding the largest share; ties go to the lowest bank;
    -1 for an empty slice), `N` [n_banks] (slices touching each bank, overlaps counted in every
    bank they touch) and `L` [n_banks] (slices homed on each bank)."""
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
    chunk = 0
    if layout == "interleaved":
        chunk = interleave_chunk(offsets, rows, cols, n_banks, elem_bytes, min_chunk_bytes)
    elif layout != "contiguous":
        raise ValueError(layout)
    bound = bank_bounds(lo, hi, n_banks)
    for s in live:
        if chunk:
            # every element's bank, counted with numpy (the same count as a Python loop)
            e = np.arange(int(offsets[s]), int(offsets[s]) + sizes[s], dtype=np.int64)
            counts[s] = np.bincount(((e - lo) // chunk) % n_banks, minlength=n_banks)
        else:
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


def weighted_shares(total, workers_per_bank, weights):
    """Targets of the weighted load balancing of Section 4.2: each bank's share of the total
    load is proportional to its number of compute units times its weight (the paper takes the
    weights in inverse proportion to latencies)."""
    prod = [float(p) * float(w) for p, w in zip(workers_per_bank, weights)]
    s = sum(prod)
    return [float(total) * q / s for q in prod]
