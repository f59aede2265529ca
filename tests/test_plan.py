"""The library's host planner, checked on the CPU (host-only plans, device -1) against the plain
checks in oracle/plan_checks.py: exactly-once coverage, balance bounds, the Section 4.1 bank
table and overlap rule, the Section 4.2 load balancer, MINIMAX on tiny instances, RR's rule,
and determinism. Topologies: MI355X-like (256 CUs / 8 XCDs), an MI300X-like part (304 / 8),
a single XCD, and odd sizes."""

import numpy as np
import pytest

import paper_2002_07062_amd as bsm
import workloads
from golden_io import paper_bank_table
from oracle import plan_checks as pc

MI355X = dict(n_cu=256, n_xcd=8, wg_per_cu=2, wg_threads=256)
TOPOLOGIES = {
    "mi355x": MI355X,
    "mi300x_like": dict(n_cu=304, n_xcd=8, wg_per_cu=2, wg_threads=256),
    "one_xcd": dict(n_cu=32, n_xcd=1, wg_per_cu=3, wg_threads=128),
    "odd": dict(n_cu=7, n_xcd=3, wg_per_cu=1, wg_threads=192),
}
ROW_COST = 64  # the library's default per-row overhead in byte equivalents


def _plan(w, schedule, topo, home=None, kclass_cols=None):
    p = bsm.bsm_plan_create(w.rows, w.cols, w.offsets[: w.batch], dtype=w.dtype,
                            schedule=schedule, topology=topo, home_xcd=home, device=-1)
    d = bsm.bsm_plan_describe(p)
    ptr, items, home_out, ov = bsm.bsm_plan_export(p)
    p.destroy()
    return d, ptr, items, home_out, ov


def _row_cost(es):
    return lambda c: ROW_COST + 2 * es * c


def _workloads():
    return {
        "c1": workloads.generate("c1"),
        "c2": workloads.generate("c2", batch=96),
        "c3": workloads.generate("c3", batch=64),
        "c4": workloads.generate("c4", batch=1024),
        "c5": workloads.generate("c5"),
        "ragged_gaps": workloads.custom([3, 0, 17, 1, 250, 9, 64], [5, 7, 1000, 2049, 64, 8, 33],
                                        gap=11, base=3),
    }


WL = _workloads()


@pytest.mark.parametrize("topo", TOPOLOGIES, ids=list(TOPOLOGIES))
@pytest.mark.parametrize("schedule", ["rr", "balanced", "xcd"])
@pytest.mark.parametrize("name", list(WL))
def test_every_row_scheduled_exactly_once(name, schedule, topo):
    w = WL[name]
    d, ptr, items, _, _ = _plan(w, schedule, TOPOLOGIES[topo])
    assert pc.check_exactly_once(ptr, items, w.offsets[: w.batch], w.rows, w.cols) == []
    t = TOPOLOGIES[topo]
    n_wg = t["n_cu"] * t["wg_per_cu"]
    # rows beyond the register tile (kernel class >= 4): 256-thread workgroups share each row,
    # so every worker is a workgroup under every schedule
    team = d["kernel_class"] >= 4
    threads = 256 if team else t["wg_threads"]
    assert d["n_wg"] == n_wg and d["wg_threads"] == threads
    per_wave = schedule != "rr" and not team
    assert d["n_workers"] == (n_wg * threads // 64 if per_wave else n_wg)
    assert d["per_wave"] == int(per_wave)
    assert d["total_rows"] == int(w.rows.sum())
    assert d["algorithmic_bytes"] == w.algorithmic_bytes
    assert d["trace_bytes"] == n_wg * (threads // 64) * 32


@pytest.mark.parametrize("name", list(WL))
def test_rr_gives_whole_slice_s_to_workgroup_s_mod_p(name):
    w = WL[name]
    d, ptr, items, _, _ = _plan(w, "rr", MI355X)
    ws, starts, _ = pc.table_row_starts(ptr, items)
    want, sl, rr, _ = pc.slice_row_starts(w.offsets[: w.batch], w.rows, w.cols)
    owner = dict(zip(starts.tolist(), ws.tolist()))
    for e, s in zip(want.tolist(), sl.tolist()):
        assert owner[e] == s % d["n_wg"]


def _unit_cost_bound(w):
    # largest cost of one tile step of the kernel: at most 16 fp32 values per lane in flight,
    # i.e. <= 64 lanes * 16 values * 2 (read + write) * 4 bytes plus its rows' overheads
    return 64 * 16 * 2 * 4 + 16 * ROW_COST + 2 * 2 * w.elem_size * int(w.cols.max())


@pytest.mark.parametrize("name", ["c2", "c3", "c4", "c5", "ragged_gaps"])
@pytest.mark.parametrize("schedule", ["balanced", "xcd"])
def test_balanced_workers_within_two_steps_of_each_other(name, schedule):
    w = WL[name]
    d, ptr, items, _, _ = _plan(w, schedule, MI355X)
    loads = pc.worker_loads(ptr, items, _row_cost(w.elem_size))
    lb = loads.sum() / len(loads)
    biggest_row = ROW_COST + 2 * w.elem_size * int(w.cols.max())
    if loads.sum() / len(loads) < 4 * _unit_cost_bound(w):
        pytest.skip("fewer tile steps than workers: balance is not the limit")
    assert loads.max() <= lb + 2 * _unit_cost_bound(w) + biggest_row, (loads.max(), lb)


def test_balanced_beats_rr_on_ragged_c5():
    w = WL["c5"]
    _, p_rr, i_rr, _, _ = _plan(w, "rr", MI355X)
    _, p_b, i_b, _, _ = _plan(w, "balanced", MI355X)
    rc = _row_cost(4)
    rr = pc.worker_loads(p_rr, i_rr, rc)
    # RR runs a whole workgroup (4 waves) per slice: compare per-wave makespans
    rr_wave = rr.max() / 4
    bal = pc.worker_loads(p_b, i_b, rc).max()
    assert bal < rr_wave / 2


@pytest.mark.parametrize("seed", range(12))
def test_tiny_instances_against_bruteforce_minimax(seed):
    """Two workers; whole-slice MINIMAX optimum by enumeration. BALANCED may split slices at
    tile steps, so its makespan must not exceed the whole-slice optimum by more than one step;
    RR can never beat the optimum."""
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 7))
    rows = rng.integers(1, 40, size=B)
    cols = rng.choice([8, 64, 200, 512], size=B)
    w = workloads.custom(rows, cols, seed=seed)
    topo = dict(n_cu=1, n_xcd=1, wg_per_cu=2, wg_threads=64)
    rc = _row_cost(4)
    costs = [int(r) * rc(int(c)) for r, c in zip(rows, cols)]
    opt, _ = pc.minimax_bruteforce(costs, 2)
    _, p_b, i_b, _, _ = _plan(w, "balanced", topo)
    bal = pc.worker_loads(p_b, i_b, rc).max()
    step = max(16 * rc(int(c)) for c in cols)  # a tile step is at most 16 rows
    assert bal <= opt + step
    assert bal >= sum(costs) / 2 - 1e-9
    _, p_r, i_r, _, _ = _plan(w, "rr", topo)
    assert pc.worker_loads(p_r, i_r, rc).max() >= opt


def test_paper_bank_table_through_the_library():
    """Section 4.1's table, reproduced by the XCD schedule with four virtual banks."""
    banks, rows = paper_bank_table()
    off = np.array([r["offset"] for r in rows], np.int64)
    R = np.array([r["R"] for r in rows], np.int32)
    C = np.array([r["C"] for r in rows], np.int32)
    p = bsm.bsm_plan_create(R, C, off, dtype="f32", schedule="xcd", device=-1,
                            topology=dict(n_cu=4, n_xcd=banks, wg_per_cu=1, wg_threads=64,
                                          flags=bsm.BSM_FLAG_CONTIGUOUS_BANKS))
    d = bsm.bsm_plan_describe(p)
    _, _, home, ov = bsm.bsm_plan_export(p)
    p.destroy()
    assert ov.tolist() == [r["overlap"] for r in rows]
    flags = np.array([r["flags"] for r in rows])
    assert d["bank_touch"] == flags.sum(axis=0).tolist()  # N_x with overlaps
    assert sum(d["bank_touch"]) > len(rows)
    assert sum(d["bank_home"]) == len(rows)                 # L_x sums to N
    assert home.tolist() == [2, 0, 1, 1, 3]
    assert d["n_overlap"] == 1


@pytest.mark.parametrize("layout,name", [("contiguous", "c1"), ("contiguous", "c5"),
                                         ("contiguous", "ragged_gaps"), ("interleaved", "c1"),
                                         ("interleaved", "c2"), ("interleaved", "c3"),
                                         ("interleaved", "c4"), ("interleaved", "c5"),
                                         ("interleaved", "ragged_gaps")])
@pytest.mark.parametrize("n_xcd", [2, 3, 8])
def test_homes_match_bruteforce_bank_table(layout, name, n_xcd):
    w = WL[name]
    if w.n_elements > 2_000_000 and (layout == "contiguous" or name == "c5"):
        w = workloads.generate("c5", batch=40)
    flags = bsm.BSM_FLAG_CONTIGUOUS_BANKS if layout == "contiguous" else 0
    topo = dict(n_cu=8 * n_xcd, n_xcd=n_xcd, wg_per_cu=1, wg_threads=64, flags=flags)
    d, ptr, items, home, ov = _plan(w, "xcd", topo)
    t = pc.bank_table(w.offsets[: w.batch], w.rows, w.cols, n_xcd, layout=layout,
                      elem_bytes=2 if w.dtype == "bf16" else 4)
    assert home.tolist() == t["home"].tolist()
    assert ov.tolist() == t["overlap"].tolist()
    assert d["bank_touch"] == t["N"].tolist()
    assert d["bank_home"] == t["L"].tolist()


@pytest.mark.parametrize("name,group", [("c2", 1), ("c3", 2), ("c4", 16)])
def test_default_banks_deal_uniform_slices_to_xcds_in_turn(name, group):
    """Interleaved banks on uniform batches: slices of 1 MiB or more (C2's fp32) are homed on
    XCD s mod 8 with no overlap, C3's 512 KiB bf16 slices in pairs and C4's 64 KiB slices in
    groups of sixteen (a 1 MiB chunk); the contiguous layout homes slice s on bank
    floor(8 s / B)."""
    w = WL[name]
    d, _, _, home, ov = _plan(w, "xcd", MI355X)
    s = np.arange(w.batch)
    assert home.tolist() == ((s // group) % 8).tolist()
    assert not ov.any() and d["n_overlap"] == 0
    assert d["moved_bytes"] == 0  # uniform slices dealt evenly: every XCD already has its share
    d, _, _, home, _ = _plan(w, "xcd", dict(MI355X, flags=bsm.BSM_FLAG_CONTIGUOUS_BANKS))
    assert home.tolist() == ((8 * s) // w.batch).tolist()
    assert d["flags"] == bsm.BSM_FLAG_CONTIGUOUS_BANKS


def _xcd_loads(w, d, ptr, items, topo, home):
    """Per-XCD cost, and the cost of rows run off their home XCD."""
    nw = topo["wg_threads"] // 64
    rc = _row_cost(w.elem_size)
    ws, starts, cols = pc.table_row_starts(ptr, items)
    want, sl, _, _ = pc.slice_row_starts(w.offsets[: w.batch], w.rows, w.cols)
    slice_of = dict(zip(want.tolist(), sl.tolist()))
    per_xcd = np.zeros(topo["n_xcd"])
    moved = 0.0
    for v, e, c in zip(ws.tolist(), starts.tolist(), cols.tolist()):
        x = (v // nw) % topo["n_xcd"]
        per_xcd[x] += rc(c)
        if home[slice_of[e]] != x:
            moved += rc(c)
    return per_xcd, moved


@pytest.mark.parametrize("pattern", ["all_on_one", "first_portion", "skewed", "virtual"])
def test_xcd_load_balancer(pattern):
    """Section 4.2: whatever the homes, after load balancing every XCD carries its share
    within about a row, and the moved load is the least any balancer must move (plus row
    rounding). 'first_portion' is the pathology where every slice is homed on the bank of its
    first byte, which puts everything on one bank."""
    w = workloads.generate("c5", batch=120)
    topo = dict(n_cu=32, n_xcd=8, wg_per_cu=1, wg_threads=128)
    rng = np.random.default_rng(3)
    home = {
        "all_on_one": np.zeros(w.batch, np.int8),
        "first_portion": np.full(w.batch, 5, np.int8),
        "skewed": rng.choice([0, 1, 2], size=w.batch).astype(np.int8),
        "virtual": None,
    }[pattern]
    d, ptr, items, home_out, _ = _plan(w, "xcd", topo, home=home)
    assert pc.check_exactly_once(ptr, items, w.offsets[: w.batch], w.rows, w.cols) == []
    per_xcd, moved = _xcd_loads(w, d, ptr, items, topo, home_out)
    share = per_xcd.sum() / topo["n_xcd"]
    biggest_row = ROW_COST + 2 * 4 * int(w.cols.max())
    assert per_xcd.max() <= share + 2 * biggest_row
    assert abs(moved - d["moved_cost"]) < 1e-6 * max(1.0, moved)
    # the balancer cuts at whole rows (midpoint rule): within half a row per XCD of the least
    # possible move, on either side
    assert abs(d["moved_cost"] - d["min_moved_cost"]) <= topo["n_xcd"] * biggest_row / 2
    loads_before = np.zeros(topo["n_xcd"])
    rc = _row_cost(4)
    for s in range(w.batch):
        loads_before[home_out[s]] += int(w.rows[s]) * rc(int(w.cols[s]))
    assert d["min_moved_cost"] == pytest.approx(
        pc.min_moved(loads_before, [loads_before.sum() / topo["n_xcd"]] * topo["n_xcd"]), abs=8)


def test_one_bank_needs_no_moves_and_matches_balanced():
    """Section 3: with the whole tensor on one bank and one XCD, the XCD schedule has nothing
    to move and balances exactly like BALANCED."""
    w = workloads.generate("c5", batch=50)
    topo = dict(n_cu=16, n_xcd=1, wg_per_cu=2, wg_threads=128)
    d_x, p_x, i_x, _, _ = _plan(w, "xcd", topo)
    d_b, p_b, i_b, _, _ = _plan(w, "balanced", topo)
    assert d_x["moved_bytes"] == 0
    assert np.array_equal(p_x, p_b) and np.array_equal(i_x, i_b)


@pytest.mark.parametrize("schedule", ["rr", "balanced", "xcd"])
def test_plans_are_deterministic(schedule):
    w = WL["c5"]
    a = _plan(w, schedule, MI355X)
    b = _plan(w, schedule, MI355X)
    for x, y in zip(a[1:], b[1:]):
        assert np.array_equal(x, y)


def test_uniform_and_explicit_offsets_give_the_same_table():
    w = WL["c2"]
    p = bsm.bsm_plan_create(512, 512, None, batch=w.batch, dtype="f32", schedule="balanced",
                            topology=MI355X, device=-1)
    a = bsm.bsm_plan_export(p)
    p.destroy()
    b = _plan(w, "balanced", MI355X)[1:]
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


def test_strided_items_fold_regular_pieces():
    """On a uniform batch every wave's pieces are equally spaced: one strided item each."""
    d, ptr, items, _, _ = _plan(WL["c2"], "balanced", MI355X)
    assert d["n_items"] == d["n_workers"]
    assert np.all(items["reps"] == d["n_rounds"])


def test_item_metadata_names_the_first_row():
    w = WL["ragged_gaps"]
    d, ptr, items, _, _ = _plan(w, "balanced", dict(n_cu=3, n_xcd=1, wg_per_cu=1, wg_threads=64))
    for it in items:
        s, r = int(it["slice"]), int(it["row_begin"])
        assert int(w.offsets[s]) + r * int(w.cols[s]) == int(it["elem_offset"])
        assert int(w.cols[s]) == int(it["cols"])


# Slices placed past 2^31 and 2^32 elements (and straddling both): the table carries 64-bit
# element offsets, and every row is still scheduled exactly once.
BIG_ROWS = [7, 5, 3, 9, 4]
BIG_COLS = [300, 1000, 4096, 64, 513]
BIG_OFFS = [(1 << 31) - 700, (1 << 31) + 12344, (1 << 32) - 3 * 4096 // 2, (1 << 32) + (1 << 20),
            (1 << 32) + (1 << 21) + 3]


@pytest.mark.parametrize("schedule", ["rr", "balanced", "xcd"])
@pytest.mark.parametrize("topo", ["mi355x", "odd"])
def test_offsets_beyond_2_32_elements(schedule, topo):
    p = bsm.bsm_plan_create(BIG_ROWS, BIG_COLS, BIG_OFFS, dtype="f32", schedule=schedule,
                            topology=TOPOLOGIES[topo], device=-1)
    d = bsm.bsm_plan_describe(p)
    ptr, items, _, _ = bsm.bsm_plan_export(p)
    p.destroy()
    assert pc.check_exactly_once(ptr, items, BIG_OFFS, BIG_ROWS, BIG_COLS) == []
    assert d["extent_elems"] == max(o + r * c for o, r, c in zip(BIG_OFFS, BIG_ROWS, BIG_COLS))
    assert int(items["elem_offset"].max()) > (1 << 32)


def _weighted_plan(w, schedule, topo, weights, home=None):
    p = bsm.bsm_plan_create(w.rows, w.cols, w.offsets[: w.batch], dtype=w.dtype,
                            schedule=schedule, topology=topo, home_xcd=home, device=-1,
                            xcd_weight=weights)
    d = bsm.bsm_plan_describe(p)
    ptr, items, home_out, ov = bsm.bsm_plan_export(p)
    p.destroy()
    return d, ptr, items, home_out, ov


@pytest.mark.parametrize("weights", [[1, 2, 3, 4, 1, 2, 3, 4], [5, 1, 1, 1, 1, 1, 1, 1],
                                     [0.25, 1, 1, 1, 1, 1, 1, 0.5]])
@pytest.mark.parametrize("pattern", ["skewed", "virtual"])
def test_weighted_load_balancing(weights, pattern):
    """Section 4.2's weighted variant: each XCD ends within about a row of its weighted share
    (workgroups x weight), and the moved load is the least any balancer must move to reach
    those shares (plus row rounding)."""
    w = workloads.generate("c5", batch=120)
    topo = dict(n_cu=32, n_xcd=8, wg_per_cu=1, wg_threads=128)
    home = None if pattern == "virtual" else \
        np.random.default_rng(4).choice([0, 1, 2], size=w.batch).astype(np.int8)
    d, ptr, items, home_out, _ = _weighted_plan(w, "xcd", topo, weights, home)
    assert pc.check_exactly_once(ptr, items, w.offsets[: w.batch], w.rows, w.cols) == []
    per_xcd, moved = _xcd_loads(w, d, ptr, items, topo, home_out)
    px = [topo["n_cu"] * topo["wg_per_cu"] // topo["n_xcd"]] * topo["n_xcd"]
    share = pc.weighted_shares(per_xcd.sum(), px, weights)
    biggest_row = ROW_COST + 2 * 4 * int(w.cols.max())
    assert np.all(np.abs(per_xcd - np.array(share)) <= 2 * biggest_row), (per_xcd, share)
    loads_before = np.zeros(topo["n_xcd"])
    rc = _row_cost(4)
    for s in range(w.batch):
        loads_before[home_out[s]] += int(w.rows[s]) * rc(int(w.cols[s]))
    least = pc.min_moved(loads_before, pc.weighted_shares(loads_before.sum(), px, weights))
    assert abs(d["moved_cost"] - least) <= topo["n_xcd"] * biggest_row / 2 + 8


def test_equal_weights_give_the_unweighted_table_and_zero_weight_gets_nothing():
    w = workloads.generate("c5", batch=100)
    _, ptr0, items0, _, _ = _plan(w, "xcd", MI355X)
    _, ptr1, items1, _, _ = _weighted_plan(w, "xcd", MI355X, [3.7] * 8)
    assert np.array_equal(ptr0, ptr1) and np.array_equal(items0, items1)
    for sch in ("rr", "balanced"):  # the weights concern the XCD schedule only
        _, p0, i0, _, _ = _plan(w, sch, MI355X)
        _, p1, i1, _, _ = _weighted_plan(w, sch, MI355X, [1, 9, 1, 9, 1, 9, 1, 9])
        assert np.array_equal(p0, p1) and np.array_equal(i0, i1)
    d, ptr, items, home, _ = _weighted_plan(w, "xcd", MI355X, [1] * 7 + [0])
    assert pc.check_exactly_once(ptr, items, w.offsets[: w.batch], w.rows, w.cols) == []
    per_xcd, _ = _xcd_loads(w, d, ptr, items, MI355X, home)
    assert per_xcd[7] == 0 and np.all(per_xcd[:7] > 0)


@pytest.mark.parametrize("weights,err", [([1] * 7 + [-1], bsm.BsmError), ([0] * 8, bsm.BsmError),
                                         ([1] * 7 + [float("nan")], bsm.BsmError),
                                         ([1] * 7, ValueError)])
def test_bad_weights_are_rejected(weights, err):
    w = workloads.generate("c1")
    with pytest.raises(err):
        _weighted_plan(w, "xcd", MI355X, weights)


@pytest.mark.parametrize("schedule", ["rr", "balanced", "xcd"])
@pytest.mark.parametrize("shape", [(384, 512, 512, 64), (384, 512, 64, 512), (7, 45, 33, 20)])
def test_gemm_plans_cover_every_output_row_in_128_row_blocks(schedule, shape):
    """Matrix-product plans: the outputs C_b are the slices; every output row is scheduled
    exactly once; workers are workgroups (512 on MI355X at two per CU), and BALANCED cuts whole
    128-row blocks, the rows a workgroup takes per round (the XCD balancer moves single rows)."""
    batch, m, n, k = shape
    p = bsm.bsm_gemm_plan_create(batch, m, n, k, "nt", "f32", schedule, topology=MI355X, device=-1)
    d = bsm.bsm_plan_describe(p)
    ptr, items, _, _ = bsm.bsm_plan_export(p)
    p.destroy()
    offs = np.arange(batch, dtype=np.int64) * m * n
    assert pc.check_exactly_once(ptr, items, offs, [m] * batch, [n] * batch) == []
    assert d["algorithmic_bytes"] == batch * (2 * (m * k + n * k) + 4 * m * n)
    assert d["per_wave"] == 0 and d["n_workers"] == 512 and d["wg_threads"] == 256
    assert d["trace_bytes"] == 512 * 4 * bsm.TRACE_DTYPE.itemsize
    if schedule == "balanced":
        # pieces are whole 128-row blocks of the row stream (batches follow each other, so a
        # block may cross into the next batch; the kernel splits it there), the stream's last
        # piece aside
        g0 = items["elem_offset"] // n
        assert np.all(g0 % 128 == 0)
        assert np.all((items["nrows"] % 128 == 0) | (g0 + items["nrows"] == batch * m))
    if shape[0] == 384 and schedule != "rr":
        # Section 6's products: 196608 output rows are 384 per workgroup, three rounds each
        rows = np.add.reduceat(items["nrows"] * items["reps"], ptr[:-1]) if len(items) else []
        assert np.all(np.asarray(rows) == 384)


@pytest.mark.parametrize("layout,n,k,wg_per_cu,one_pass", [
    ("nt_softmax", 512, 64, 0, True), ("nt_softmax", 72, 8, 0, True), ("nt_softmax", 520, 64, 0, False),
    ("nt_softmax", 64, 64, 0, False), ("nt_softmax", 512, 72, 0, True), ("nt_softmax", 512, 128, 0, True),
    ("nt_softmax", 512, 136, 0, False), ("nt_softmax", 512, 0, 0, False),
    ("nt_softmax", 512, 64, 3, False), ("nt_softmax", 512, 64, 1, True), ("nt", 512, 64, 0, False)])
def test_score_softmax_plans_pick_the_one_pass_form(layout, n, k, wg_per_cu, one_pass):
    """The score product with the row softmax runs in one pass for 0 < k <= 128 and
    64 < n <= 512 unless the topology asks for three or more workgroups per CU: such plans
    default to two workgroups per CU and cut BALANCED pieces at 64-row blocks (the rows a
    workgroup takes per round); the others default to three per CU and 128-row blocks."""
    batch, m = 6, 512
    topo = dict(n_cu=256, n_xcd=8, wg_per_cu=wg_per_cu, wg_threads=256)
    p = bsm.bsm_gemm_plan_create(batch, m, n, k, layout, "bf16", "balanced", topology=topo, device=-1)
    d = bsm.bsm_plan_describe(p)
    ptr, items, _, _ = bsm.bsm_plan_export(p)
    p.destroy()
    assert d["n_wg"] == 256 * (wg_per_cu or (2 if one_pass else 3))
    if n == 0:
        return
    unit = 64 if one_pass else 128
    g0 = items["elem_offset"] // n
    assert np.all(g0 % unit == 0)
    assert np.all((items["nrows"] % unit == 0) | (g0 + items["nrows"] == batch * m))
    assert np.any(items["nrows"] % 128 != 0) == one_pass


def test_gemm_plan_rejects_bad_arguments():
    for args in [(-1, 4, 4, 4, 0), (1, -4, 4, 4, 0), (1, 4, 4, 4, 3)]:
        with pytest.raises(bsm.BsmError) as e:
            bsm.bsm_gemm_plan_create(*args[:4], layout=args[4], topology=MI355X, device=-1)
        assert e.value.status == bsm.BSM_ERR_INVALID_ARG
    # layout 2 is the score product with the row softmax
    bsm.bsm_gemm_plan_create(1, 4, 4, 4, layout=2, topology=MI355X, device=-1).destroy()
    # a matrix-product plan does not run as a softmax, nor a softmax plan as a product
    lib = bsm.load()
    import ctypes
    g = bsm.bsm_gemm_plan_create(2, 8, 8, 8, topology=MI355X, device=-1)
    assert lib.bsm_plan_execute(g.handle, ctypes.c_void_p(16), ctypes.c_void_p(4096), None, None) == bsm.BSM_ERR_UNSUPPORTED
    g.destroy()
    s = bsm.bsm_plan_create([4], [4], [0], dtype="f32", topology=MI355X, device=-1)
    assert lib.bsm_gemm_execute(s.handle, ctypes.c_void_p(16), ctypes.c_void_p(16), ctypes.c_void_p(4096),
                                1.0, None, None) == bsm.BSM_ERR_UNSUPPORTED
    s.destroy()
    # one-shot: no-ops and validation before any GPU call
    assert lib.bsm_gemm(None, None, None, 0, 4, 4, 4, 0, 0, 1.0, 0, None) == bsm.BSM_OK
    assert lib.bsm_gemm(None, None, None, 2, 4, 4, 4, 0, 0, 1.0, 0, None) == bsm.BSM_ERR_INVALID_ARG
    assert lib.bsm_gemm(None, None, None, 2, 4, 4, 4, 5, 0, 1.0, 0, None) == bsm.BSM_ERR_INVALID_ARG


@pytest.mark.parametrize("seed", range(60))
def test_random_geometries_every_row_exactly_once(seed):
    """Randomized geometries (slices in random order with gaps, empty slices, widths from 1 to
    9000) on random topologies, under every schedule and with random homes for XCD: every row
    is scheduled exactly once and the plan's totals are the geometry's."""
    from random_geometry import geometry, topology

    w = geometry(seed)
    topo = topology(seed)
    rng = np.random.default_rng(20_000 + seed)
    for schedule in ("rr", "balanced", "xcd"):
        home = None
        if schedule == "xcd" and rng.random() < 0.5 and w.batch:
            home = rng.integers(0, topo["n_xcd"], size=w.batch).astype(np.int8)
        d, ptr, items, _, _ = _plan(w, schedule, topo, home=home)
        assert pc.check_exactly_once(ptr, items, w.offsets[: w.batch], w.rows, w.cols) == [], (seed, schedule)
        assert d["total_rows"] == int(w.rows.sum())
        assert d["algorithmic_bytes"] == 2 * 4 * int(np.sum(w.rows.astype(np.int64) * w.cols))
        assert d["n_wg"] == topo["n_cu"] * topo["wg_per_cu"]
        if schedule == "xcd":
            assert sum(d["xcd_bytes"][: topo["n_xcd"]]) == d["algorithmic_bytes"]
