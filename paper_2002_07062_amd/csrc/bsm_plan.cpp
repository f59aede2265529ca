// Host planner for the batched row softmax: builds the per-worker work table.
//
// The paper's scheduler (Sections 3-5) maps patches (slices) to compute clusters and builds the
// mapping table once, up front.  Here the table is a CSR list of row ranges per worker, built
// on the host once per geometry.  A worker is a workgroup (RR) or a single wave (BALANCED and
// XCD).
//
// Cost model (Section 4.2's execution time E_t, for a bandwidth-bound kernel): a row of C
// elements costs row_cost + 2*C*elem_bytes byte equivalents (read once, written once); each
// work item adds item_cost (reported, not balanced).  Cuts use exact integer arithmetic.
//
// BALANCED and XCD cut a team's row stream into rounds, and every round into one piece per
// worker.  All workers of a team then sweep the stream together, so at any moment the team
// touches one compact window of memory (DRAM rows stay open; measured on MI355X to be worth
// ~20% over one contiguous chunk per worker), while each worker's total stays balanced.
#include "bsm_plan.hpp"

#include <algorithm>
#include <chrono>
#include <cmath>
#include <limits>
#include <numeric>

#include "bsm_tile.hpp"

namespace bsm {
namespace {

using i128 = __int128;

constexpr int64_t kMaxElems = int64_t(1) << 60;
constexpr int64_t kMaxBins = int64_t(1) << 26;
constexpr int kLongRowKernelClass = 4;  // the kernel class that runs rows beyond the register tile

// Rows [0, nrows) of row length `cols`; row r starts at element off + r * cols.
struct Span {
    int64_t off;
    int32_t cols;
    int32_t nrows;
};

int64_t row_cost_of(const Topology& t, int elem_bytes, int32_t cols) {
    return static_cast<int64_t>(std::llround(t.row_cost)) + static_cast<int64_t>(cols) * 2 * elem_bytes;
}

// Appends a span, merging it into the previous one when it continues it in memory with the
// same row length (adjacent slices of equal C form one longer run of rows).
void push_span(std::vector<Span>* v, Span s) {
    if (s.nrows <= 0) return;
    if (!v->empty()) {
        Span& b = v->back();
        if (b.cols == s.cols && b.off + static_cast<int64_t>(b.nrows) * b.cols == s.off &&
            static_cast<int64_t>(b.nrows) + s.nrows <= std::numeric_limits<int32_t>::max()) {
            b.nrows += s.nrows;
            return;
        }
    }
    v->push_back(s);
}

// A stream segment of n_units equal units of unit_rows rows, each costing unit_cost.
struct Segment {
    int64_t off;
    int32_t cols;
    int32_t unit_rows;
    int64_t n_units;
    int64_t unit_cost;
};

std::vector<Segment> segments_of(const std::vector<Span>& stream, const Topology& t, int es,
                                 int kernel_class, bool whole_steps) {
    std::vector<Segment> segs;
    for (const Span& s : stream) {
        const int64_t rc = row_cost_of(t, es, s.cols);
        const int32_t unit = !whole_steps ? 1
                             : t.row_unit > 0 ? t.row_unit
                                              : std::max(1, wave_step_rows(s.cols, es, kernel_class));
        const int64_t full = s.nrows / unit, tail = s.nrows % unit;
        if (full > 0) segs.push_back(Segment{s.off, s.cols, unit, full, unit * rc});
        if (tail > 0)
            segs.push_back(Segment{s.off + full * unit * static_cast<int64_t>(s.cols), s.cols,
                                   static_cast<int32_t>(tail), 1, tail * rc});
    }
    return segs;
}

// Cuts the stream into K consecutive bins with costs proportional to `weights` (all equal when
// empty), at unit boundaries.  A unit occupying cost interval [a, a + c) of the total T goes to
// the bin whose cumulative-weight interval holds its scaled midpoint: the largest j with
// cw[j] <= W (a + c/2) / T.  Every bin is then within one unit's cost of its share; bins of
// zero weight get nothing.
void cut_stream(const std::vector<Segment>& segs, const std::vector<int64_t>& weights, int64_t K,
                std::vector<std::vector<Span>>* bins) {
    bins->assign(static_cast<size_t>(K), {});
    if (K <= 0) return;
    std::vector<i128> cw(static_cast<size_t>(K) + 1, 0);
    for (int64_t j = 0; j < K; ++j)
        cw[j + 1] = cw[j] + (weights.empty() ? 1 : std::max<int64_t>(0, weights[j]));
    const i128 W = cw[K];
    i128 T = 0;
    for (const Segment& s : segs) T += static_cast<i128>(s.n_units) * s.unit_cost;
    if (T == 0 || W == 0) return;

    i128 A0 = 0;  // stream cost before the current segment
    for (const Segment& s : segs) {
        const i128 c = s.unit_cost;
        // Unit u's midpoint scaled by 2W: pos(u) = W (2 A0 + (2u + 1) c); its bin is the
        // largest j with 2 T cw[j] <= pos(u).
        auto bin_of = [&](int64_t u) -> int64_t {
            const i128 pos = W * (2 * A0 + (2 * static_cast<i128>(u) + 1) * c);
            int64_t lo = 0, hi = K - 1;
            while (lo < hi) {
                const int64_t mid = (lo + hi + 1) / 2;
                if (2 * T * cw[mid] <= pos) lo = mid; else hi = mid - 1;
            }
            return lo;
        };
        int64_t u = 0;
        while (u < s.n_units) {
            const int64_t b = bin_of(u);
            int64_t u_end = s.n_units;
            if (b + 1 < K) {
                // first unit v with W (2 A0 + (2v + 1) c) >= 2 T cw[b+1]
                const i128 need = 2 * T * cw[b + 1] - W * (2 * A0 + c);
                const i128 den = 2 * W * c;
                i128 v = need <= 0 ? 0 : (need + den - 1) / den;
                if (v < u + 1) v = u + 1;
                if (v < u_end) u_end = static_cast<int64_t>(v);
            }
            const int64_t r0 = u * s.unit_rows;
            const int64_t nr = (u_end - u) * s.unit_rows;
            push_span(&(*bins)[b], Span{s.off + r0 * s.cols, s.cols, static_cast<int32_t>(nr)});
            u = u_end;
        }
        A0 += static_cast<i128>(s.n_units) * c;
    }
}

i128 span_cost(const Span& s, const Topology& t, int es) {
    return static_cast<i128>(s.nrows) * row_cost_of(t, es, s.cols);
}

// Rounds for one team: the stream is cut into n_rounds * W bins of equal cost (whole tile
// steps of the kernel where possible); in each round the largest pieces go to the workers
// with the least accumulated cost (ties to the lower worker), which keeps every worker's total
// within about one piece-granule of the others.
int64_t assign_rounds(const std::vector<Span>& stream, const std::vector<int32_t>& workers,
                      const Topology& t, int es, int kernel_class,
                      std::vector<std::vector<Span>>* per_worker) {
    const int64_t W = static_cast<int64_t>(workers.size());
    if (W == 0 || stream.empty()) return 0;
    i128 total = 0;
    for (const Span& s : stream) total += span_cost(s, t, es);
    const std::vector<Segment> segs = segments_of(stream, t, es, kernel_class, true);
    int64_t n_units = 0;
    for (const Segment& s : segs) n_units += s.n_units;
    // Rounds of about W * piece_bytes each, but never so many that a piece falls below one
    // tile step of the kernel.
    const double per_round = static_cast<double>(W) * std::max(1, t.piece_bytes);
    int64_t n_rounds = static_cast<int64_t>(std::llround(static_cast<double>(total) / per_round));
    n_rounds = std::min<int64_t>(n_rounds, n_units / W);
    n_rounds = std::max<int64_t>(1, std::min<int64_t>(n_rounds, kMaxBins / W));
    std::vector<std::vector<Span>> bins;
    cut_stream(segs, {}, n_rounds * W, &bins);

    std::vector<i128> acc(static_cast<size_t>(W), 0);
    std::vector<i128> cost(static_cast<size_t>(W));
    std::vector<int64_t> ob(static_cast<size_t>(W)), ow(static_cast<size_t>(W));
    for (int64_t r = 0; r < n_rounds; ++r) {
        for (int64_t k = 0; k < W; ++k) {
            i128 c = 0;
            for (const Span& s : bins[r * W + k]) c += span_cost(s, t, es);
            cost[k] = c;
        }
        std::iota(ob.begin(), ob.end(), 0);
        std::iota(ow.begin(), ow.end(), 0);
        std::stable_sort(ob.begin(), ob.end(), [&](int64_t a, int64_t b) { return cost[a] > cost[b]; });
        std::stable_sort(ow.begin(), ow.end(), [&](int64_t a, int64_t b) { return acc[a] < acc[b]; });
        for (int64_t k = 0; k < W; ++k) {
            const int64_t slot = ow[k], bin = ob[k];
            acc[slot] += cost[bin];
            for (const Span& s : bins[r * W + bin]) push_span(&(*per_worker)[workers[slot]], s);
        }
    }
    return n_rounds;
}

// Elements of [a, b) (relative to the span's start) that fall in each of n banks when the
// span is cut into chunks of g elements dealt to the banks in turn (chunk k -> bank k mod n).
void interleaved_shares(int64_t a, int64_t b, int64_t g, int n, std::vector<int64_t>* share) {
    share->assign(static_cast<size_t>(n), 0);
    const int64_t ka = a / g, kb = (b - 1) / g;
    if (ka == kb) {
        (*share)[ka % n] += b - a;
        return;
    }
    (*share)[ka % n] += (ka + 1) * g - a;
    (*share)[kb % n] += b - kb * g;
    const int64_t whole = kb - ka - 1;  // full chunks between the two partial ones
    for (int j = 0; j < n; ++j) (*share)[j] += (whole / n) * g;
    for (int64_t j = 0; j < whole % n; ++j) (*share)[(ka + 1 + j) % n] += g;
}

}  // namespace

int64_t bank_chunk_elems(const Geometry& g, int n, bool contiguous) {
    int64_t lo = std::numeric_limits<int64_t>::max(), hi = 0, live = 0;
    for (int64_t s = 0; s < g.batch; ++s) {
        const int64_t sz = static_cast<int64_t>(g.R[s]) * g.C[s];
        if (sz == 0) continue;
        lo = std::min(lo, g.off[s]);
        hi = std::max(hi, g.off[s] + sz);
        ++live;
    }
    if (contiguous || live == 0 || hi <= lo) return 0;
    const int64_t span = hi - lo;
    const int64_t mean = std::max<int64_t>(1, span / live);
    const int64_t min_elems = (kBankChunkBytes + g.elem_bytes - 1) / g.elem_bytes;
    const int64_t chunk = mean * ((min_elems + mean - 1) / mean);
    // a span of no more than n chunks keeps the contiguous banks (one range per bank)
    if (static_cast<i128>(chunk) * n >= span) return 0;
    return chunk;
}

namespace {

// Homes of Section 4.1 over virtual banks that partition the span [lo, hi) of the non-empty
// slices: chunks of bank_chunk_elems() elements dealt to the banks in turn, or n equal
// contiguous ranges (chunk 0).  A slice's home is the bank holding its largest share (lowest
// index on a tie), and OVERLAP is set when it has elements in two or more banks.
void assign_homes(const Geometry& g, int n, bool contiguous, const int8_t* user, Table* tab) {
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
    const int64_t chunk = bank_chunk_elems(g, n, contiguous);
    std::vector<int64_t> bound(static_cast<size_t>(n) + 1);
    for (int b = 0; b <= n; ++b)
        bound[b] = lo + static_cast<int64_t>(static_cast<i128>(b) * (hi - lo) / n);
    std::vector<int64_t> share(static_cast<size_t>(n));
    for (int64_t s = 0; s < B; ++s) {
        const int64_t o = g.off[s], e = o + static_cast<int64_t>(g.R[s]) * g.C[s];
        if (e == o) continue;
        if (chunk > 0) {
            interleaved_shares(o - lo, e - lo, chunk, n, &share);
        } else {
            for (int b = 0; b < n; ++b)
                share[b] = std::max<int64_t>(0, std::min(e, bound[b + 1]) - std::max(o, bound[b]));
        }
        int best = -1, touched = 0;
        for (int b = 0; b < n; ++b) {
            if (share[b] <= 0) continue;
            ++touched;
            st.bank_touch[b] += 1;
            if (best < 0 || share[b] > share[best]) best = b;
        }
        tab->home[s] = static_cast<int8_t>(best);
        tab->overlap[s] = touched > 1 ? 1 : 0;
        st.n_overlap += touched > 1 ? 1 : 0;
        st.bank_home[best] += 1;
    }
}

struct Piece {  // rows [row_begin, row_begin + nrows) of slice `slice`
    int32_t slice;
    int32_t row_begin;
    int32_t nrows;
};

// XCD schedule, steps 1 and 2: homes, then the load balancer.  Returns each XCD's row stream.
std::vector<std::vector<Span>> xcd_streams(const Geometry& g, const Topology& t,
                                           const int8_t* user_home, Table* tab) {
    const int n = t.n_xcd;
    const int P = t.n_wg();
    const int es = g.elem_bytes;
    assign_homes(g, n, t.contiguous_banks, user_home, tab);

    std::vector<int64_t> Px(static_cast<size_t>(n), 0);
    for (int w = 0; w < P; ++w) Px[w % n] += 1;

    std::vector<std::vector<Piece>> own(static_cast<size_t>(n));
    std::vector<i128> load(static_cast<size_t>(n), 0);
    i128 total = 0;
    for (int64_t s = 0; s < g.batch; ++s) {
        if (g.R[s] == 0 || g.C[s] == 0) continue;
        const int x = tab->home[s];
        own[x].push_back(Piece{static_cast<int32_t>(s), 0, g.R[s]});
        const i128 c = static_cast<i128>(g.R[s]) * row_cost_of(t, es, g.C[s]);
        load[x] += c;
        total += c;
    }
    // Share of XCD x: total * Px Wx / sum(Py Wy), with Px its workgroups and Wx its weight
    // (Section 4.2's weighted balancing; all weights equal unless the caller gives them).
    std::vector<i128> Wx(static_cast<size_t>(n));
    i128 wsum = 0;
    for (int x = 0; x < n; ++x) {
        Wx[x] = static_cast<i128>(Px[x]) * (t.xcd_weight.empty() ? 1 : t.xcd_weight[x]);
        wsum += Wx[x];
    }
    std::vector<i128> share(static_cast<size_t>(n));
    for (int x = 0; x < n; ++x) share[x] = total * Wx[x] / wsum;
    double min_moved = 0.0;
    for (int x = 0; x < n; ++x)
        if (load[x] > share[x]) min_moved += static_cast<double>(load[x] - share[x]);
    tab->stats.min_moved_cost = min_moved;

    // Over-loaded XCDs keep the rows whose cost midpoint lies within their share; the rest
    // joins a pool that goes to the under-loaded XCDs in proportion to their deficits.
    std::vector<std::vector<Piece>> kept(static_cast<size_t>(n));
    std::vector<Piece> pool;
    for (int x = 0; x < n; ++x) {
        if (load[x] <= share[x]) {
            kept[x] = own[x];
            continue;
        }
        i128 A0 = 0;
        for (const Piece& p : own[x]) {
            const i128 c = row_cost_of(t, es, g.C[p.slice]);
            const i128 num = 2 * share[x] - 2 * A0 - c;  // rows rr with 2(A0 + rr c) + c <= 2 share
            int64_t keep = 0;
            if (num >= 0) keep = static_cast<int64_t>(std::min<i128>(num / (2 * c) + 1, p.nrows));
            if (keep > 0) kept[x].push_back(Piece{p.slice, p.row_begin, static_cast<int32_t>(keep)});
            if (keep < p.nrows)
                pool.push_back(Piece{p.slice, p.row_begin + static_cast<int32_t>(keep),
                                     static_cast<int32_t>(p.nrows - keep)});
            A0 += static_cast<i128>(p.nrows) * c;
        }
    }
    std::vector<std::vector<Span>> stream(static_cast<size_t>(n));
    auto to_span = [&](const Piece& p) {
        return Span{g.off[p.slice] + static_cast<int64_t>(p.row_begin) * g.C[p.slice], g.C[p.slice], p.nrows};
    };
    for (int x = 0; x < n; ++x)
        for (const Piece& p : kept[x]) push_span(&stream[x], to_span(p));
    if (!pool.empty()) {
        std::vector<int64_t> deficit(static_cast<size_t>(n), 0);
        bool any = false;
        for (int x = 0; x < n; ++x) {
            if (load[x] < share[x]) {
                deficit[x] = static_cast<int64_t>(share[x] - load[x]);
                any = any || deficit[x] > 0;
            }
        }
        if (!any) {  // rounding left no deficit: the least loaded XCD per weight takes it
            int best = -1;
            for (int x = 0; x < n; ++x)
                if (Wx[x] > 0 && (best < 0 || load[x] * Wx[best] < load[best] * Wx[x])) best = x;
            deficit[best] = 1;
        }
        std::vector<Span> pool_spans;
        double moved_cost = 0.0;
        int64_t moved_bytes = 0;
        for (const Piece& p : pool) {
            pool_spans.push_back(to_span(p));  // unmerged: each piece keeps its own cost
            moved_cost += static_cast<double>(p.nrows) * row_cost_of(t, es, g.C[p.slice]);
            moved_bytes += static_cast<int64_t>(p.nrows) * g.C[p.slice] * 2 * es;
        }
        std::vector<std::vector<Span>> recv;
        cut_stream(segments_of(pool_spans, t, es, 0, false), deficit, n, &recv);
        for (int x = 0; x < n; ++x)
            for (const Span& s : recv[x]) push_span(&stream[x], s);
        tab->stats.moved_cost = moved_cost;
        tab->stats.moved_bytes = moved_bytes;
        // Each XCD takes its rows in memory order, received ones included, so that the eight
        // XCDs sweep the tensor together instead of ending on rows scattered over it.
        for (int x = 0; x < n; ++x) {
            std::vector<Span> v = std::move(stream[x]);
            std::sort(v.begin(), v.end(), [](const Span& a, const Span& b) { return a.off < b.off; });
            stream[x].clear();
            for (const Span& sp : v) push_span(&stream[x], sp);
        }
    }
    return stream;
}

// Locates the slice holding element `e` (which lies inside some non-empty slice).
struct SliceIndex {
    std::vector<std::pair<int64_t, int32_t>> starts;  // (offset, slice), non-empty slices
    explicit SliceIndex(const Geometry& g) {
        for (int64_t s = 0; s < g.batch; ++s)
            if (g.R[s] > 0 && g.C[s] > 0) starts.emplace_back(g.off[s], static_cast<int32_t>(s));
        std::sort(starts.begin(), starts.end());
    }
    int32_t find(int64_t e) const {
        auto it = std::upper_bound(starts.begin(), starts.end(),
                                   std::make_pair(e, std::numeric_limits<int32_t>::max()));
        return (it == starts.begin()) ? -1 : std::prev(it)->second;
    }
};

// Turns a worker's spans into items, folding runs of equal-length, equally spaced spans into
// one strided item.
void emit_items(const Geometry& g, const SliceIndex& idx, const std::vector<Span>& spans,
                std::vector<bsm_item>* items) {
    size_t i = 0;
    while (i < spans.size()) {
        const Span& a = spans[i];
        int64_t reps = 1, stride = 0;
        if (i + 1 < spans.size()) {
            const Span& b = spans[i + 1];
            const int64_t d = b.off - a.off;
            if (b.cols == a.cols && b.nrows == a.nrows && d > 0 && d % a.cols == 0 &&
                d / a.cols <= std::numeric_limits<int32_t>::max()) {
                stride = d / a.cols;
                reps = 2;
                while (i + reps < spans.size()) {
                    const Span& c = spans[i + reps];
                    const Span& p = spans[i + reps - 1];
                    if (c.cols != a.cols || c.nrows != a.nrows || c.off - p.off != d ||
                        reps >= std::numeric_limits<int32_t>::max())
                        break;
                    ++reps;
                }
            }
        }
        bsm_item it;
        it.elem_offset = a.off;
        it.cols = a.cols;
        it.nrows = a.nrows;
        it.reps = static_cast<int32_t>(reps);
        it.rep_stride = static_cast<int32_t>(stride);
        it.slice = idx.find(a.off);
        it.row_begin = it.slice >= 0 ? static_cast<int32_t>((a.off - g.off[it.slice]) / g.C[it.slice]) : 0;
        items->push_back(it);
        i += static_cast<size_t>(reps);
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

bool quick_geometry(const int64_t* slice_offsets, const int32_t* rows, const int32_t* cols,
                    int64_t batch, int64_t* extent) {
    *extent = 0;
    if (batch < 0 || batch > std::numeric_limits<int32_t>::max()) return false;
    if (batch == 0) return true;
    if (!rows || !cols) return false;
    if (!slice_offsets) {
        const int64_t R = rows[0], C = cols[0];
        if (R < 0 || C < 0) return false;
        const int64_t per = R * C;
        if (per > 0 && batch > kMaxElems / per) return false;
        *extent = per * batch;
        return true;
    }
    int64_t end = 0;  // end of the previous non-empty slice
    for (int64_t s = 0; s < batch; ++s) {
        if (rows[s] < 0 || cols[s] < 0 || slice_offsets[s] < 0) return false;
        const int64_t sz = static_cast<int64_t>(rows[s]) * cols[s];
        if (sz > kMaxElems || slice_offsets[s] > kMaxElems - sz) return false;
        if (sz == 0) continue;
        if (slice_offsets[s] < end) return false;  // out of order, or overlapping
        end = slice_offsets[s] + sz;
    }
    *extent = end;
    return true;
}

std::string check_topology(const Topology& t) {
    if (t.n_cu < 1 || t.n_cu > 65536) return "n_cu out of range";
    if (t.n_xcd < 1 || t.n_xcd > BSM_MAX_XCD) return "n_xcd out of range [1, 16]";
    if (t.wg_per_cu < 1 || t.wg_per_cu > 64) return "wg_per_cu out of range [1, 64]";
    if (t.wg_threads < 64 || t.wg_threads > 1024 || t.wg_threads % 64 != 0)
        return "wg_threads must be a multiple of 64 in [64, 1024]";
    if (static_cast<int64_t>(t.n_cu) * t.wg_per_cu * (t.wg_threads / 64) > (1 << 22))
        return "too many waves";
    if (t.piece_bytes < 1 || t.piece_bytes > (1 << 30)) return "piece_bytes out of range";
    if (!(t.item_cost >= 0.0) || !(t.row_cost >= 0.0) || !std::isfinite(t.item_cost) ||
        !std::isfinite(t.row_cost) || t.row_cost > 1e12 || t.item_cost > 1e12)
        return "cost model values must be finite and >= 0";
    if (!t.xcd_weight.empty()) {
        if (static_cast<int>(t.xcd_weight.size()) != t.n_xcd) return "xcd_weight needs n_xcd entries";
        int64_t with_workers = 0;
        for (int x = 0; x < t.n_xcd; ++x) {
            if (t.xcd_weight[x] < 0 || t.xcd_weight[x] > (int64_t(1) << 30))
                return "xcd_weight out of range";
            if (x < t.n_wg()) with_workers += t.xcd_weight[x];
        }
        if (with_workers == 0) return "xcd_weight gives every XCD with workgroups weight 0";
    }
    return "";
}

std::string build_table(const Geometry& g, bsm_schedule schedule, const Topology& t,
                        const int8_t* home_xcd, int kernel_class, Table* tab) {
    const auto t0 = std::chrono::steady_clock::now();
    const int P = t.n_wg();
    const int nw = t.waves_per_wg();
    const int es = g.elem_bytes;
    *tab = Table{};
    bsm_plan_stats& st = tab->stats;
    if (home_xcd && schedule == BSM_SCHED_XCD) {
        for (int64_t s = 0; s < g.batch; ++s)
            if (home_xcd[s] < 0 || home_xcd[s] >= t.n_xcd)
                return "home_xcd[" + std::to_string(s) + "] outside [0, n_xcd)";
    }
    std::vector<std::vector<Span>> per_worker;
    int64_t rounds = 0;
    switch (schedule) {
        case BSM_SCHED_RR: {
            tab->per_wave = false;
            per_worker.assign(static_cast<size_t>(P), {});
            for (int64_t s = 0; s < g.batch; ++s)
                if (g.R[s] > 0 && g.C[s] > 0)
                    per_worker[static_cast<size_t>(s % P)].push_back(Span{g.off[s], g.C[s], g.R[s]});
            tab->home.assign(static_cast<size_t>(g.batch), -1);
            tab->overlap.assign(static_cast<size_t>(g.batch), 0);
            break;
        }
        case BSM_SCHED_BALANCED: {
            tab->per_wave = true;
            per_worker.assign(static_cast<size_t>(P) * nw, {});
            std::vector<Span> stream;
            for (int64_t s = 0; s < g.batch; ++s)
                if (g.R[s] > 0 && g.C[s] > 0) push_span(&stream, Span{g.off[s], g.C[s], g.R[s]});
            // Order of the workers within a round, chosen by measurement on MI355X: for rows
            // in a register tile, XCD-major (each XCD takes one contiguous part of every round:
            // +7% on 16384 x 128 x 128, equal elsewhere); for long rows, workgroup order
            // (consecutive pieces on consecutive workgroups, hence alternating XCDs: +8%).
            std::vector<int32_t> workers;
            workers.reserve(static_cast<size_t>(P) * nw);
            if (kernel_class >= kLongRowKernelClass) {
                for (int v = 0; v < P * nw; ++v) workers.push_back(v);
            } else {
                for (int x = 0; x < t.n_xcd; ++x)
                    for (int w = x; w < P; w += t.n_xcd)
                        for (int k = 0; k < nw; ++k) workers.push_back(w * nw + k);
            }
            rounds = assign_rounds(stream, workers, t, es, kernel_class, &per_worker);
            tab->home.assign(static_cast<size_t>(g.batch), -1);
            tab->overlap.assign(static_cast<size_t>(g.batch), 0);
            break;
        }
        case BSM_SCHED_XCD: {
            tab->per_wave = true;
            per_worker.assign(static_cast<size_t>(P) * nw, {});
            const std::vector<std::vector<Span>> streams = xcd_streams(g, t, home_xcd, tab);
            for (int x = 0; x < t.n_xcd; ++x) {
                std::vector<int32_t> workers;
                for (int w = x; w < P; w += t.n_xcd)
                    for (int k = 0; k < nw; ++k) workers.push_back(w * nw + k);
                rounds = std::max(rounds, assign_rounds(streams[x], workers, t, es, kernel_class, &per_worker));
            }
            break;
        }
        default:
            return "unknown schedule";
    }

    // CSR pack + statistics.
    const SliceIndex idx(g);
    const int64_t n_workers = static_cast<int64_t>(per_worker.size());
    tab->worker_ptr.assign(static_cast<size_t>(n_workers) + 1, 0);
    double max_cost = 0.0, sum_cost = 0.0;
    for (int64_t v = 0; v < n_workers; ++v) {
        const size_t first = tab->items.size();
        emit_items(g, idx, per_worker[v], &tab->items);
        if (tab->items.size() > static_cast<size_t>(std::numeric_limits<int32_t>::max()))
            return "work table exceeds 2^31 items";
        double cost = 0.0;
        const int x = static_cast<int>((tab->per_wave ? v / nw : v) % t.n_xcd);
        for (size_t i = first; i < tab->items.size(); ++i) {
            const bsm_item& it = tab->items[i];
            const int64_t rows = static_cast<int64_t>(it.nrows) * it.reps;
            cost += t.item_cost + static_cast<double>(rows) * row_cost_of(t, es, it.cols);
            st.xcd_bytes[x] += rows * it.cols * 2 * es;
        }
        tab->worker_ptr[v + 1] = static_cast<int32_t>(tab->items.size());
        max_cost = std::max(max_cost, cost);
        sum_cost += cost;
    }
    double max_row = 0.0;
    for (int64_t s = 0; s < g.batch; ++s)
        if (g.R[s] > 0 && g.C[s] > 0)
            max_row = std::max(max_row, static_cast<double>(row_cost_of(t, es, g.C[s])));

    st.batch = g.batch;
    st.n_items = static_cast<int64_t>(tab->items.size());
    st.total_rows = g.total_rows;
    st.algorithmic_bytes = g.total_elems * 2 * es;
    st.extent_elems = g.extent;
    st.n_rounds = rounds;
    st.n_workers = static_cast<int32_t>(n_workers);
    st.per_wave = tab->per_wave ? 1 : 0;
    st.n_wg = P;
    st.n_xcd = t.n_xcd;
    st.wg_threads = t.wg_threads;
    st.schedule = schedule;
    st.max_cols = g.max_cols;
    st.max_worker_cost = max_cost;
    st.mean_worker_cost = n_workers ? sum_cost / static_cast<double>(n_workers) : 0.0;
    st.max_row_cost = max_row;
    st.trace_bytes = static_cast<int64_t>(P) * nw * static_cast<int64_t>(sizeof(bsm_trace_rec));
    st.build_us = std::chrono::duration<double, std::micro>(std::chrono::steady_clock::now() - t0).count();
    return "";
}

}  // namespace bsm
