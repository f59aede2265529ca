// Host planner for the batched row softmax: builds the per-workgroup work table.
//
// The paper's scheduler (Sections 3-5) maps patches (slices) to compute clusters.  Here a
// cluster is a persistent workgroup, the table is a CSR list of row ranges per workgroup, and
// it is built once per geometry on the host (the paper's "constructed upfront" table).
//
// Cost model (Section 4.2's E_t, for a bandwidth-bound kernel): a row of C elements costs
// row_cost + 2*C*elem_bytes (read once, write once) byte equivalents; every work item adds
// item_cost.  All cuts are made at row boundaries with exact integer arithmetic.
#include "bsm_plan.hpp"

#include <algorithm>
#include <chrono>
#include <cmath>
#include <limits>

namespace bsm {
namespace {

using i128 = __int128;

constexpr int64_t kMaxElems = int64_t(1) << 60;

struct Piece {
    int32_t slice;
    int32_t row_begin;
    int32_t nrows;
};

int64_t row_cost_of(const Geometry& g, const Topology& t, int32_t s) {
    return static_cast<int64_t>(std::llround(t.row_cost)) +
           static_cast<int64_t>(g.C[s]) * 2 * g.elem_bytes;
}

void push_merged(std::vector<Piece>* bin, Piece p) {
    if (p.nrows <= 0) return;
    if (!bin->empty()) {
        Piece& last = bin->back();
        if (last.slice == p.slice && last.row_begin + last.nrows == p.row_begin) {
            last.nrows += p.nrows;
            return;
        }
    }
    bin->push_back(p);
}

// Cuts the row stream `pieces` (rows taken in order) into K consecutive ranges whose costs are
// proportional to `weights` (all equal when `weights` is empty).  A row occupying cost
// interval [a, a + c) of the stream's total T goes to the bin whose cumulative-weight interval
// contains its midpoint scaled to the weights: bin j with cw[j] <= W(a + c/2)/T < cw[j+1].
// Each bin's cost is then within one row's cost of its share.  Zero-weight bins get nothing.
void cut_stream(const Geometry& g, const Topology& t, const std::vector<Piece>& pieces,
                const std::vector<int64_t>& weights, int K, std::vector<std::vector<Piece>>* bins) {
    bins->assign(static_cast<size_t>(K), {});
    if (K <= 0) return;
    std::vector<i128> cw(static_cast<size_t>(K) + 1, 0);
    for (int j = 0; j < K; ++j)
        cw[j + 1] = cw[j] + (weights.empty() ? 1 : std::max<int64_t>(0, weights[j]));
    const i128 W = cw[K];
    i128 T = 0;
    for (const Piece& p : pieces) T += static_cast<i128>(p.nrows) * row_cost_of(g, t, p.slice);
    if (T == 0 || W == 0) return;

    i128 A0 = 0;  // stream cost before the current piece
    for (const Piece& p : pieces) {
        const i128 c = row_cost_of(g, t, p.slice);
        // Row rr's midpoint scaled by 2W: pos(rr) = W*(2*A0 + (2rr+1)c); it belongs to the
        // largest bin j with 2T*cw[j] <= pos(rr).
        auto bin_of = [&](int64_t rr) -> int {
            const i128 pos = W * (2 * A0 + (2 * static_cast<i128>(rr) + 1) * c);
            // largest j with 2T*cw[j] <= pos
            int lo = 0, hi = K - 1;
            while (lo < hi) {
                const int mid = (lo + hi + 1) / 2;
                if (2 * T * cw[mid] <= pos) lo = mid; else hi = mid - 1;
            }
            return lo;
        };
        int64_t r = 0;
        while (r < p.nrows) {
            const int b = bin_of(r);
            int64_t r_end = p.nrows;
            if (b + 1 < K) {
                // first row rr with W*(2*A0 + (2rr+1)c) >= 2T*cw[b+1]
                const i128 need = 2 * T * cw[b + 1] - W * (2 * A0 + c);
                const i128 den = 2 * W * c;
                i128 rr = need <= 0 ? 0 : (need + den - 1) / den;
                if (rr < r + 1) rr = r + 1;
                if (rr < r_end) r_end = static_cast<int64_t>(rr);
            }
            push_merged(&(*bins)[b], Piece{p.slice, p.row_begin + static_cast<int32_t>(r),
                                           static_cast<int32_t>(r_end - r)});
            r = r_end;
        }
        A0 += static_cast<i128>(p.nrows) * c;
    }
}

std::vector<Piece> whole_slices(const Geometry& g) {
    std::vector<Piece> v;
    for (int64_t s = 0; s < g.batch; ++s)
        if (g.R[s] > 0 && g.C[s] > 0) v.push_back(Piece{static_cast<int32_t>(s), 0, g.R[s]});
    return v;
}

// Homes of Section 4.1.  Virtual banks: n equal contiguous element ranges over the span of the
// non-empty slices; a slice's home is the bank holding its largest share (lowest index on a
// tie), OVERLAP is set when it has elements in two or more banks.
void assign_homes(const Geometry& g, int n, const int8_t* user, Table* tab) {
    const int64_t B = g.batch;
    tab->home.assign(static_cast<size_t>(B), -1);
    tab->overlap.assign(static_cast<size_t>(B), 0);
    bsm_plan_stats& st = tab->stats;
    if (user) {
        for (int64_t s = 0; s < B; ++s) {
            if (g.R[s] == 0 || g.C[s] == 0) continue;
            tab->home[s] = user[s];
            st.bank_touch[user[s]] += 1;
            st.bank_home[user[s]] += 1;
        }
        return;
    }
    int64_t lo = std::numeric_limits<int64_t>::max(), hi = 0;
    for (int64_t s = 0; s < B; ++s) {
        const int64_t sz = static_cast<int64_t>(g.R[s]) * g.C[s];
        if (sz == 0) continue;
        lo = std::min(lo, g.off[s]);
        hi = std::max(hi, g.off[s] + sz);
    }
    if (hi <= lo) return;
    std::vector<int64_t> bound(static_cast<size_t>(n) + 1);
    for (int b = 0; b <= n; ++b)
        bound[b] = lo + static_cast<int64_t>(static_cast<i128>(b) * (hi - lo) / n);
    for (int64_t s = 0; s < B; ++s) {
        const int64_t o = g.off[s], e = o + static_cast<int64_t>(g.R[s]) * g.C[s];
        if (e == o) continue;
        // first bank whose end is past o
        int b0 = static_cast<int>(std::upper_bound(bound.begin() + 1, bound.end(), o) -
                                  (bound.begin() + 1));
        int best = -1, touched = 0;
        int64_t best_share = -1;
        for (int b = b0; b < n && bound[b] < e; ++b) {
            const int64_t share = std::min(e, bound[b + 1]) - std::max(o, bound[b]);
            if (share <= 0) continue;
            ++touched;
            st.bank_touch[b] += 1;
            if (share > best_share) {
                best_share = share;
                best = b;
            }
        }
        tab->home[s] = static_cast<int8_t>(best);
        tab->overlap[s] = touched > 1 ? 1 : 0;
        st.n_overlap += touched > 1 ? 1 : 0;
        st.bank_home[best] += 1;
    }
}

// Schedule XCD: homes, then load balancing across XCDs, then equal-cost cuts per XCD.
void plan_xcd(const Geometry& g, const Topology& t, const int8_t* user_home, Table* tab,
              std::vector<std::vector<Piece>>* bins) {
    const int n = t.n_xcd;
    const int P = t.n_wg();
    assign_homes(g, n, user_home, tab);

    std::vector<int> Px(static_cast<size_t>(n), 0);
    for (int w = 0; w < P; ++w) Px[w % n] += 1;

    std::vector<std::vector<Piece>> own(static_cast<size_t>(n));
    std::vector<i128> load(static_cast<size_t>(n), 0);
    i128 total = 0;
    for (int64_t s = 0; s < g.batch; ++s) {
        if (g.R[s] == 0 || g.C[s] == 0) continue;
        const int x = tab->home[s];
        own[x].push_back(Piece{static_cast<int32_t>(s), 0, g.R[s]});
        const i128 c = static_cast<i128>(g.R[s]) * row_cost_of(g, t, static_cast<int32_t>(s));
        load[x] += c;
        total += c;
    }
    // Fair share of XCD x: total * Px / P (XCDs differ only in how many workgroups they run).
    std::vector<i128> share(static_cast<size_t>(n));
    for (int x = 0; x < n; ++x) share[x] = total * Px[x] / P;

    double min_moved = 0.0;
    for (int x = 0; x < n; ++x)
        if (load[x] > share[x]) min_moved += static_cast<double>(load[x] - share[x]);
    tab->stats.min_moved_cost = min_moved;

    // Over-loaded XCDs keep rows whose midpoint lies within their share; the rest join a pool.
    std::vector<std::vector<Piece>> stream(static_cast<size_t>(n));
    std::vector<Piece> pool;
    for (int x = 0; x < n; ++x) {
        if (load[x] <= share[x]) {
            stream[x] = own[x];
            continue;
        }
        i128 A0 = 0;
        for (const Piece& p : own[x]) {
            const i128 c = row_cost_of(g, t, p.slice);
            // rows rr with 2*(A0 + rr*c) + c <= 2*share are kept
            const i128 num = 2 * share[x] - 2 * A0 - c;
            int64_t keep = 0;
            if (num >= 0) keep = static_cast<int64_t>(std::min<i128>(num / (2 * c) + 1, p.nrows));
            if (keep > 0) push_merged(&stream[x], Piece{p.slice, p.row_begin, static_cast<int32_t>(keep)});
            if (keep < p.nrows)
                pool.push_back(Piece{p.slice, p.row_begin + static_cast<int32_t>(keep),
                                     static_cast<int32_t>(p.nrows - keep)});
            A0 += static_cast<i128>(p.nrows) * c;
        }
    }
    // The pool is split over the under-loaded XCDs in proportion to their deficits.
    std::vector<int64_t> deficit(static_cast<size_t>(n), 0);
    bool any = false;
    for (int x = 0; x < n; ++x) {
        if (load[x] < share[x]) {
            deficit[x] = static_cast<int64_t>(share[x] - load[x]);
            any = any || deficit[x] > 0;
        }
    }
    if (!pool.empty()) {
        if (!any) {  // rounding left no deficit: give the pool to the least loaded XCD with WGs
            int best = -1;
            for (int x = 0; x < n; ++x)
                if (Px[x] > 0 && (best < 0 || load[x] * Px[best] < load[best] * Px[x])) best = x;
            deficit[best] = 1;
        }
        std::vector<std::vector<Piece>> recv;
        cut_stream(g, t, pool, deficit, n, &recv);
        for (int x = 0; x < n; ++x)
            for (const Piece& p : recv[x]) push_merged(&stream[x], p);
        double moved_cost = 0.0;
        int64_t moved_bytes = 0;
        for (const Piece& p : pool) {
            moved_cost += static_cast<double>(p.nrows) * row_cost_of(g, t, p.slice);
            moved_bytes += static_cast<int64_t>(p.nrows) * g.C[p.slice] * 2 * g.elem_bytes;
        }
        tab->stats.moved_cost = moved_cost;
        tab->stats.moved_bytes = moved_bytes;
    }
    // Within each XCD, equal-cost cut over its workgroups w = x, x + n, x + 2n, ...
    bins->assign(static_cast<size_t>(P), {});
    for (int x = 0; x < n; ++x) {
        if (Px[x] == 0) continue;
        std::vector<std::vector<Piece>> local;
        cut_stream(g, t, stream[x], {}, Px[x], &local);
        for (int l = 0; l < Px[x]; ++l) (*bins)[static_cast<size_t>(x) + static_cast<size_t>(l) * n] = std::move(local[l]);
    }
}

}  // namespace

std::string make_geometry(const int64_t* slice_offsets, const int32_t* rows, const int32_t* cols,
                          int64_t batch, int elem_bytes, Geometry* g) {
    if (batch < 0) return "batch is negative";
    if (batch > std::numeric_limits<int32_t>::max()) return "batch exceeds 2^31 - 1 slices";
    g->batch = batch;
    g->elem_bytes = elem_bytes;
    g->off.assign(static_cast<size_t>(batch), 0);
    g->R.assign(static_cast<size_t>(batch), 0);
    g->C.assign(static_cast<size_t>(batch), 0);
    g->extent = g->total_rows = g->total_elems = 0;
    g->max_cols = 0;
    if (batch == 0) return "";
    if (!rows || !cols) return "rows or cols is NULL";
    if (!slice_offsets) {
        const int64_t R = rows[0], C = cols[0];
        if (R < 0 || C < 0) return "rows[0] or cols[0] is negative";
        const int64_t per = R * C;
        if (per > 0 && batch > kMaxElems / per) return "uniform geometry exceeds 2^60 elements";
        for (int64_t s = 0; s < batch; ++s) {
            g->off[s] = s * per;
            g->R[s] = static_cast<int32_t>(R);
            g->C[s] = static_cast<int32_t>(C);
        }
    } else {
        std::vector<std::pair<int64_t, int64_t>> spans;
        spans.reserve(static_cast<size_t>(batch));
        for (int64_t s = 0; s < batch; ++s) {
            if (rows[s] < 0 || cols[s] < 0) return "rows[" + std::to_string(s) + "] or cols[] is negative";
            if (slice_offsets[s] < 0) return "slice_offsets[" + std::to_string(s) + "] is negative";
            const int64_t sz = static_cast<int64_t>(rows[s]) * cols[s];
            if (sz > kMaxElems || slice_offsets[s] > kMaxElems - sz)
                return "slice " + std::to_string(s) + " ends beyond 2^60 elements";
            g->off[s] = slice_offsets[s];
            g->R[s] = rows[s];
            g->C[s] = cols[s];
            if (sz > 0) spans.emplace_back(slice_offsets[s], slice_offsets[s] + sz);
        }
        std::sort(spans.begin(), spans.end());
        for (size_t i = 1; i < spans.size(); ++i)
            if (spans[i].first < spans[i - 1].second)
                return "two slices overlap (element " + std::to_string(spans[i].first) + ")";
    }
    for (int64_t s = 0; s < batch; ++s) {
        const int64_t sz = static_cast<int64_t>(g->R[s]) * g->C[s];
        if (sz == 0) continue;
        g->extent = std::max(g->extent, g->off[s] + sz);
        g->total_rows += g->R[s];
        g->total_elems += sz;
        g->max_cols = std::max(g->max_cols, g->C[s]);
    }
    return "";
}

std::string check_topology(const Topology& t) {
    if (t.n_cu < 1 || t.n_cu > 65536) return "n_cu out of range";
    if (t.n_xcd < 1 || t.n_xcd > BSM_MAX_XCD) return "n_xcd out of range [1, 16]";
    if (t.wg_per_cu < 1 || t.wg_per_cu > 64) return "wg_per_cu out of range [1, 64]";
    if (static_cast<int64_t>(t.n_cu) * t.wg_per_cu > (1 << 22)) return "too many workgroups";
    if (t.wg_threads < 64 || t.wg_threads > 1024 || t.wg_threads % 64 != 0)
        return "wg_threads must be a multiple of 64 in [64, 1024]";
    if (!(t.item_cost >= 0.0) || !(t.row_cost >= 0.0) || !std::isfinite(t.item_cost) ||
        !std::isfinite(t.row_cost) || t.row_cost > 1e12 || t.item_cost > 1e12)
        return "cost model values must be finite and >= 0";
    return "";
}

std::string build_table(const Geometry& g, bsm_schedule schedule, const Topology& t,
                        const int8_t* home_xcd, Table* tab) {
    const auto t0 = std::chrono::steady_clock::now();
    const int P = t.n_wg();
    *tab = Table{};
    bsm_plan_stats& st = tab->stats;
    std::vector<std::vector<Piece>> bins;

    if (home_xcd && schedule == BSM_SCHED_XCD) {
        for (int64_t s = 0; s < g.batch; ++s)
            if (home_xcd[s] < 0 || home_xcd[s] >= t.n_xcd)
                return "home_xcd[" + std::to_string(s) + "] outside [0, n_xcd)";
    }
    switch (schedule) {
        case BSM_SCHED_RR: {
            bins.assign(static_cast<size_t>(P), {});
            for (const Piece& p : whole_slices(g)) bins[static_cast<size_t>(p.slice % P)].push_back(p);
            tab->home.assign(static_cast<size_t>(g.batch), -1);
            tab->overlap.assign(static_cast<size_t>(g.batch), 0);
            break;
        }
        case BSM_SCHED_BALANCED: {
            cut_stream(g, t, whole_slices(g), {}, P, &bins);
            tab->home.assign(static_cast<size_t>(g.batch), -1);
            tab->overlap.assign(static_cast<size_t>(g.batch), 0);
            break;
        }
        case BSM_SCHED_XCD:
            plan_xcd(g, t, home_xcd, tab, &bins);
            break;
        default:
            return "unknown schedule";
    }

    // CSR pack + statistics.
    int64_t n_items = 0;
    for (const auto& b : bins) n_items += static_cast<int64_t>(b.size());
    if (n_items > std::numeric_limits<int32_t>::max()) return "work table exceeds 2^31 items";
    tab->wg_ptr.assign(static_cast<size_t>(P) + 1, 0);
    tab->items.reserve(static_cast<size_t>(n_items));
    double max_cost = 0.0, sum_cost = 0.0;
    for (int w = 0; w < P; ++w) {
        double cost = 0.0;
        for (const Piece& p : bins[w]) {
            bsm_item it;
            it.elem_offset = g.off[p.slice] + static_cast<int64_t>(p.row_begin) * g.C[p.slice];
            it.cols = g.C[p.slice];
            it.nrows = p.nrows;
            it.slice = p.slice;
            it.row_begin = p.row_begin;
            tab->items.push_back(it);
            cost += t.item_cost + static_cast<double>(p.nrows) * row_cost_of(g, t, p.slice);
            st.xcd_bytes[w % t.n_xcd] += static_cast<int64_t>(p.nrows) * g.C[p.slice] * 2 * g.elem_bytes;
        }
        tab->wg_ptr[w + 1] = static_cast<int32_t>(tab->items.size());
        max_cost = std::max(max_cost, cost);
        sum_cost += cost;
    }
    double max_row = 0.0;
    for (int64_t s = 0; s < g.batch; ++s)
        if (g.R[s] > 0 && g.C[s] > 0)
            max_row = std::max(max_row, static_cast<double>(row_cost_of(g, t, static_cast<int32_t>(s))));

    st.batch = g.batch;
    st.n_items = n_items;
    st.total_rows = g.total_rows;
    st.algorithmic_bytes = g.total_elems * 2 * g.elem_bytes;
    st.extent_elems = g.extent;
    st.n_wg = P;
    st.n_xcd = t.n_xcd;
    st.wg_threads = t.wg_threads;
    st.schedule = schedule;
    st.max_cols = g.max_cols;
    st.max_wg_cost = max_cost;
    st.mean_wg_cost = P ? sum_cost / P : 0.0;
    st.max_row_cost = max_row;
    st.trace_bytes = static_cast<int64_t>(P) * (t.wg_threads / 64) * static_cast<int64_t>(sizeof(bsm_trace_rec));
    st.build_us = std::chrono::duration<double, std::micro>(std::chrono::steady_clock::now() - t0).count();
    return "";
}

}  // namespace bsm
