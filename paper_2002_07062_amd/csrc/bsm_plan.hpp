// Host planner: slice geometry -> per-worker work table (CSR), for the three schedules.
// Pure C++17, no HIP runtime calls.  The paper's HW batch scheduler (Section 5) in software.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "bsm.h"

namespace bsm {

struct Geometry {
    int64_t batch = 0;
    std::vector<int64_t> off;  // [batch] element offset of slice s
    std::vector<int32_t> R;    // [batch]
    std::vector<int32_t> C;    // [batch]
    int elem_bytes = 4;        // in and out share the element type
    int64_t extent = 0;        // max over slices of off + R*C (0 if all empty)
    int64_t total_rows = 0;
    int64_t total_elems = 0;
    int32_t max_cols = 0;
};

struct Topology {
    int32_t n_cu = 256;
    int32_t n_xcd = 8;
    int32_t wg_per_cu = 2;
    int32_t wg_threads = 256;
    int32_t piece_bytes = 8192;  // traffic per worker piece in one round
    double item_cost = 1024.0;   // byte equivalents
    double row_cost = 64.0;      // byte equivalents on top of the row's bytes
    // Weighted load balancing (Section 4.2): relative weight of each XCD's share under the XCD
    // schedule, e.g. in inverse proportion to a measured latency.  Empty = equal weights.
    std::vector<int64_t> xcd_weight;
    // Rows per cutting unit (0: the softmax register-tile step for the row's length).  The
    // matrix-product kernels take rows 32 at a time.
    int32_t row_unit = 0;
    // XCD schedule: virtual banks as n_xcd equal contiguous ranges instead of interleaved chunks
    bool contiguous_banks = false;
    int32_t n_wg() const { return n_cu * wg_per_cu; }
    int32_t waves_per_wg() const { return wg_threads / 64; }
};

struct Table {
    std::vector<int32_t> worker_ptr;  // [n_workers + 1]
    std::vector<bsm_item> items;
    std::vector<int8_t> home;         // [batch]; -1 where the schedule assigns no home
    std::vector<uint8_t> overlap;     // [batch]
    bool per_wave = false;
    bsm_plan_stats stats{};
};

// Smallest chunk of the interleaved virtual banks of the XCD schedule.  Measured on MI355X: with
// chunks of at least this size (and at least one mean slice) the eight XCDs stream neighbouring
// memory at any moment, each XCD about one round of its workers (256 waves x 4 KiB of input)
// inside one chunk, and the XCD schedule runs within 1.5% of BALANCED on cold uniform data;
// eight contiguous banks, one window per XCD ~1/8 of the batch apart, cost 4-13%, and 256 KiB
// chunks (one XCD round spread over eight chunks) 3-12% on 16384 x 128 x 128 fp32.
constexpr int64_t kBankChunkBytes = 1024 * 1024;

// Chunk, in elements, of the interleaved virtual banks for `g` over n banks: the mean extent of a
// non-empty slice times the smallest factor that makes it at least kBankChunkBytes.  0 means n
// equal contiguous ranges: asked for, or the span of the slices holds no more than n chunks.
int64_t bank_chunk_elems(const Geometry& g, int n, bool contiguous);

// Checks the geometry (sizes, overflow, slices not overlapping) and fills `g`.  Returns an
// empty string on success, else what is wrong.
std::string make_geometry(const int64_t* slice_offsets, const int32_t* rows,
                          const int32_t* cols, int64_t batch, int elem_bytes, Geometry* g);

// Allocation-free check of the common case, for calls that repeat a geometry: true, with the
// extent, when the geometry is valid and its non-empty slices lie in ascending offset order;
// false when make_geometry must decide (an error, or slices out of order).
bool quick_geometry(const int64_t* slice_offsets, const int32_t* rows, const int32_t* cols,
                    int64_t batch, int64_t* extent);

std::string check_topology(const Topology& t);

// Builds the table for `schedule`.  home_xcd may be null.  kernel_class is the register-tile
// class of the kernel that will run the table (pieces are sized in whole tile steps).
// Returns "" or an error message.
std::string build_table(const Geometry& g, bsm_schedule schedule, const Topology& t,
                        const int8_t* home_xcd, int kernel_class, Table* out);

}  // namespace bsm
