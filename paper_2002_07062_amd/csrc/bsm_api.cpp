// C-ABI of libbsm.so: argument checks, plans (host table + device copy), the one-shot plan
// cache, device queries and the copy reference.  Every failure is a status code plus a
// thread-local message; nothing is thrown across the ABI.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <list>
#include <memory>
#include <mutex>
#include <new>
#include <string>
#include <thread>
#include <vector>

#include "bsm.h"
#include "bsm_launch.hpp"
#include "bsm_plan.hpp"
#include "bsm_tile.hpp"

struct bsm_plan_s {
    int device = -1;  // -1: host-only plan
    bsm_dtype dtype = BSM_F32;
    bsm_schedule schedule = BSM_SCHED_RR;
    bsm::Topology topo;
    bsm::Geometry geo;
    bsm::Table table;
    int kernel_class = 0;
    bool shifted = false;  // some slice's rows do not start and end on 16-byte vectors
    // A matrix-product plan (bsm_gemm_plan_create) instead of a softmax plan: the slices are
    // the outputs C_b (gemm_m x gemm_n), A_b is gemm_m x gemm_k, layout 0 = NT, 1 = NN,
    // 2 = NT with the row softmax of the products.
    bool gemm = false;
    int gemm_m = 0, gemm_n = 0, gemm_k = 0, gemm_layout = 0;
    bool gemm_single = false;  // layout 2 in one pass (products held in registers)
    int64_t gemm_batch = 0;
    int lds_floats_per_wave = 0;  // one-wave long-row staging (kernel classes 4, 5 on a device)
    int32_t flags = 0;            // BSM_FLAG_* bits
    void* d_table = nullptr;  // device copy: worker_ptr, then items (256-byte aligned)
    const int32_t* d_worker_ptr = nullptr;
    const bsm_item* d_items = nullptr;
    std::atomic<bool> used{false};  // executed at least once (destroy then waits for the device)
    // One-shot cache plans only (all under the cache lock except `inflight`):
    bool pooled = false;              // d_table is a buffer of the cache's pool, not owned
    size_t table_cap = 0;             // bytes of that buffer
    std::atomic<int> inflight{0};     // calls between lookup and the end of their launch
    std::vector<hipStream_t> streams; // streams the plan ran on (up to kMaxTrackedStreams)
    bool many_streams = false;        // ran on more streams than are tracked
    bool captured = false;            // launched into a graph capture: never evicted
    hipStream_t upload_stream = nullptr;
    hipEvent_t upload_done = nullptr; // recorded after the table upload
    bool uploaded = false;            // upload_done seen complete
};

namespace {

thread_local std::string g_error;

bsm_status fail(bsm_status st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_error = buf;
    return st;
}

bsm_status hip_fail(hipError_t e, const char* what) {
    return fail(BSM_ERR_HIP, "%s: %s (%d)", what, hipGetErrorString(e), static_cast<int>(e));
}

// Restores the caller's current device on scope exit.
struct DeviceGuard {
    int prev = -1;
    bool switched = false;
    hipError_t enter(int device) {
        hipError_t e = hipGetDevice(&prev);
        if (e != hipSuccess) return e;
        if (prev != device) {
            e = hipSetDevice(device);
            if (e != hipSuccess) return e;
            switched = true;
        }
        return hipSuccess;
    }
    ~DeviceGuard() {
        if (switched) (void)hipSetDevice(prev);
    }
};

// Waves per CU that measured fastest on MI355X: 8 for fp32 rows (more waves only add DRAM
// page conflicts), 16 for bf16 rows, which carry twice the ALU work per byte and need the
// extra waves to overlap it with memory.  Plans with rows beyond the register tile run two
// 256-thread workgroups per CU (8 waves), each holding one or two rows in its registers.
constexpr int kLongRowClass = 4;
int default_waves_per_cu(bsm_dtype d, int kclass) {
    if (kclass >= kLongRowClass) return 8;
    return d == BSM_BF16 ? 16 : 8;
}

// Smallest LDS region worth staging a row in (shorter rows never reach the long-row path).
constexpr int64_t kMinStageBytes = 8192;

// LDS per wave for long-row staging: the CU's LDS split over its resident workgroups, capped
// by the per-workgroup limit, less the kernels' own static LDS (`static_bytes` per workgroup),
// split over the waves and rounded down to 64 bytes.
int64_t lds_bytes_per_wave(const hipDeviceProp_t& prop, const bsm::Topology& t,
                           int64_t static_bytes) {
    const int64_t per_cu = static_cast<int64_t>(prop.maxSharedMemoryPerMultiProcessor);
    const int64_t per_wg = std::min<int64_t>(per_cu / std::max(1, t.wg_per_cu),
                                             static_cast<int64_t>(prop.sharedMemPerBlock)) -
                           static_bytes;
    const int64_t per_wave = (per_wg / t.waves_per_wg()) & ~static_cast<int64_t>(63);
    return per_wave >= kMinStageBytes ? per_wave : 0;
}
constexpr int kDefaultPieceBytes = 8192;
constexpr float kDefaultItemCost = 1024.0f;
constexpr float kDefaultRowCost = 64.0f;

int elem_bytes_of(bsm_dtype d) { return d == BSM_BF16 ? 2 : 4; }

// Whether some non-empty slice's rows do not all start and end on 16-byte vectors.
bool any_shifted(const bsm::Geometry& g) {
    const int64_t epv = bsm::kVecBytes / g.elem_bytes;
    for (int64_t s = 0; s < g.batch; ++s)
        if (g.R[s] > 0 && g.C[s] > 0 && ((g.off[s] | static_cast<int64_t>(g.C[s])) % epv) != 0)
            return true;
    return false;
}

bool valid_dtype(int d) { return d == BSM_F32 || d == BSM_BF16; }
bool valid_schedule(int s) { return s == BSM_SCHED_RR || s == BSM_SCHED_BALANCED || s == BSM_SCHED_XCD; }

// Defaults for a device: all CUs, the runtime's XCD count, 256-thread workgroups.  wg_per_cu
// is left 0: a plan picks it from the element type (default_waves_per_cu), capped by the
// occupancy of the kernel instance it launches, so the persistent grid is always fully
// resident and the static table is what actually runs.
bsm_status default_topology(int device, bsm_topology* t) {
    hipDeviceProp_t prop;
    hipError_t e = hipGetDeviceProperties(&prop, device);
    if (e != hipSuccess) return hip_fail(e, "hipGetDeviceProperties");
    int n_xcd = 1;
    e = hipDeviceGetAttribute(&n_xcd, hipDeviceAttributeNumberOfXccs, device);
    if (e != hipSuccess || n_xcd < 1) n_xcd = 1;
    if (n_xcd > BSM_MAX_XCD) n_xcd = BSM_MAX_XCD;
    std::memset(t, 0, sizeof *t);
    t->n_cu = prop.multiProcessorCount;
    t->n_xcd = n_xcd;
    t->wg_threads = 256;
    t->wg_per_cu = 0;
    t->piece_bytes = kDefaultPieceBytes;
    t->item_cost = kDefaultItemCost;
    t->row_cost = kDefaultRowCost;
    return BSM_OK;
}

bsm_status resolve_topology(const bsm_topology* user, int device, bsm_dtype dtype, int kclass,
                            bool shifted, bsm::Topology* out) {
    bsm_topology t;
    if (device >= 0) {
        bsm_status st = default_topology(device, &t);
        if (st != BSM_OK) return st;
    } else {
        std::memset(&t, 0, sizeof t);
        t.n_cu = 256;
        t.n_xcd = 8;
        t.wg_threads = 256;
        t.piece_bytes = kDefaultPieceBytes;
        t.item_cost = kDefaultItemCost;
        t.row_cost = kDefaultRowCost;
    }
    if (user) {
        if ((user->flags & ~(BSM_FLAG_TEMPORAL | BSM_FLAG_CONTIGUOUS_BANKS)) != 0)
            return fail(BSM_ERR_INVALID_ARG, "topology.flags has unknown bits 0x%x", user->flags);
        if (user->n_cu < 0 || user->n_xcd < 0 || user->wg_per_cu < 0 || user->wg_threads < 0 ||
            user->piece_bytes < 0)
            return fail(BSM_ERR_INVALID_ARG, "topology fields must be >= 0 (0 = default)");
        if (user->n_cu > 0) t.n_cu = user->n_cu;
        if (user->n_xcd > 0) t.n_xcd = user->n_xcd;
        if (user->wg_per_cu > 0) t.wg_per_cu = user->wg_per_cu;
        if (user->wg_threads > 0) t.wg_threads = user->wg_threads;
        if (user->piece_bytes > 0) t.piece_bytes = user->piece_bytes;
        if (user->item_cost > 0.0f) t.item_cost = user->item_cost;
        if (user->row_cost > 0.0f) t.row_cost = user->row_cost;
    }
    if (t.wg_per_cu <= 0 && t.wg_threads >= 64) {
        const int want = std::max(1, default_waves_per_cu(dtype, kclass) / (t.wg_threads / 64));
        t.wg_per_cu = want;
        if (device >= 0 && t.wg_threads <= 1024 && t.wg_threads % 64 == 0) {
            int n = 0;
            DeviceGuard g;
            hipError_t e = g.enter(device);
            hipDeviceProp_t prop;
            if (e == hipSuccess) e = hipGetDeviceProperties(&prop, device);
            size_t lds = 0;
            if (e == hipSuccess && kclass >= kLongRowClass) {
                bsm::Topology probe;
                probe.wg_per_cu = want;
                probe.wg_threads = t.wg_threads;
                int static_bytes = 0;
                e = bsm::static_lds_bytes(dtype, kclass, shifted, &static_bytes);
                if (e == hipSuccess)
                    lds = static_cast<size_t>(lds_bytes_per_wave(prop, probe, static_bytes)) *
                          (t.wg_threads / 64);
            }
            if (e == hipSuccess)
                e = bsm::resident_wgs_per_cu(dtype, kclass, shifted, t.wg_threads, lds, &n);
            if (e != hipSuccess) return hip_fail(e, "occupancy query");
            t.wg_per_cu = std::max(1, std::min(want, n));
        }
    }
    out->n_cu = t.n_cu;
    out->n_xcd = t.n_xcd;
    out->wg_per_cu = t.wg_per_cu;
    out->wg_threads = t.wg_threads;
    out->piece_bytes = t.piece_bytes;
    out->item_cost = t.item_cost;
    out->row_cost = t.row_cost;
    out->contiguous_banks = user && (user->flags & BSM_FLAG_CONTIGUOUS_BANKS) != 0;
    std::string err = bsm::check_topology(*out);
    if (!err.empty()) return fail(BSM_ERR_INVALID_ARG, "topology: %s", err.c_str());
    return BSM_OK;
}

void free_device(bsm_plan p) {
    if (p->device < 0 || p->pooled) return;  // a pooled table belongs to the one-shot cache
    DeviceGuard g;
    if (g.enter(p->device) != hipSuccess) return;
    // Executions on any stream may still be reading the table.  (Nothing is recorded per
    // execution: an event after every launch costs the stream a gap of several microseconds
    // between kernels.)
    if (p->used) (void)hipDeviceSynchronize();
    if (p->d_table) {
        (void)hipFree(p->d_table);
        p->d_table = nullptr;
    }
}

// Caller weights (any positive scale) -> integer weights with the largest at 2^30.
bsm_status resolve_weights(const float* w, bsm::Topology* t) {
    t->xcd_weight.clear();
    if (!w) return BSM_OK;
    float mx = 0.0f;
    for (int x = 0; x < t->n_xcd; ++x) {
        if (!std::isfinite(w[x]) || w[x] < 0.0f)
            return fail(BSM_ERR_INVALID_ARG, "xcd_weight[%d] = %g: weights must be finite and >= 0", x,
                        static_cast<double>(w[x]));
        mx = std::max(mx, w[x]);
    }
    if (!(mx > 0.0f)) return fail(BSM_ERR_INVALID_ARG, "xcd_weight: every weight is 0");
    for (int x = 0; x < t->n_xcd; ++x)
        t->xcd_weight.push_back(static_cast<int64_t>(std::llround(static_cast<double>(w[x]) / mx * 1073741824.0)));
    return BSM_OK;
}

// Device layout of a work table: the worker row pointer, then the items at the next 256-byte
// boundary.
size_t table_items_at(const bsm::Table& t) {
    return (t.worker_ptr.size() * sizeof(int32_t) + 255) & ~static_cast<size_t>(255);
}
size_t table_bytes(const bsm::Table& t) {
    return table_items_at(t) + std::max<size_t>(t.items.size(), 1) * sizeof(bsm_item);
}

// Test hook for the allocation-failure paths: the environment variable BSM_TEST_ALLOC_FAIL set
// to "host" makes plan creation fail as if a host allocation had failed (after the table is
// built, so everything built so far must be released), "device" as if the work table's device
// allocation had failed.  Read at every plan creation.
enum class AllocFail { none, host, device };
AllocFail alloc_fail_hook() {
    const char* v = std::getenv("BSM_TEST_ALLOC_FAIL");
    if (!v) return AllocFail::none;
    if (std::strcmp(v, "host") == 0) return AllocFail::host;
    if (std::strcmp(v, "device") == 0) return AllocFail::device;
    return AllocFail::none;
}

hipError_t table_malloc(void** ptr, size_t bytes) {
    if (alloc_fail_hook() == AllocFail::device) {
        *ptr = nullptr;
        return hipErrorOutOfMemory;
    }
    return hipMalloc(ptr, bytes);
}

// upload == false (one-shot cache misses): the table stays on the host; the cache uploads it
// asynchronously into a buffer of its pool.
bsm_status create_plan(bsm_plan* out_plan, const int64_t* offs, const int32_t* rows,
                       const int32_t* cols, int64_t batch, bsm_dtype dtype, bsm_schedule schedule,
                       const int8_t* home_xcd, const float* xcd_weight,
                       const bsm_topology* topology, int device, int32_t row_unit = 0,
                       bool product = false, bool upload = true) {
    if (!out_plan) return fail(BSM_ERR_INVALID_ARG, "out_plan is NULL");
    *out_plan = nullptr;
    if (!valid_dtype(dtype)) return fail(BSM_ERR_INVALID_ARG, "unknown dtype %d", static_cast<int>(dtype));
    if (!valid_schedule(schedule)) return fail(BSM_ERR_INVALID_ARG, "unknown schedule %d", static_cast<int>(schedule));
    if (device < -1) return fail(BSM_ERR_INVALID_ARG, "device %d", device);
    if (device == -1 && !topology) return fail(BSM_ERR_INVALID_ARG, "a host-only plan (device -1) needs a topology");
    if (device >= 0) {
        int n = 0;
        hipError_t e = hipGetDeviceCount(&n);
        if (e != hipSuccess) return hip_fail(e, "hipGetDeviceCount");
        if (device >= n) return fail(BSM_ERR_INVALID_ARG, "device %d of %d", device, n);
    }
    std::unique_ptr<bsm_plan_s> p(new (std::nothrow) bsm_plan_s);
    if (!p) return fail(BSM_ERR_OOM, "plan allocation failed");
    bsm_topology tu{};  // the caller's topology with a long-row plan's workgroup size
    try {
        std::string err = bsm::make_geometry(offs, rows, cols, batch, elem_bytes_of(dtype), &p->geo);
        if (!err.empty()) return fail(BSM_ERR_INVALID_ARG, "geometry: %s", err.c_str());
        p->shifted = any_shifted(p->geo);
        p->kernel_class = bsm::kernel_class_for(p->geo.max_cols, elem_bytes_of(dtype), p->shifted);
        // Rows beyond the register tile are worked by whole workgroups (team_threads of the
        // class), one row at a time: such plans run that workgroup size whatever the topology
        // asks (a row's bits depend on it), and every worker of their table is a workgroup.
        const bool team = !product && p->kernel_class >= kLongRowClass;
        if (team) {
            if (topology) tu = *topology;
            tu.wg_threads = bsm::team_threads(p->kernel_class);
            topology = &tu;
        }
        // bf16 plans of class 3 run in instances compiled for workgroups of up to 256 threads
        if (!product && dtype == BSM_BF16 && p->kernel_class == 3 && topology &&
            topology->wg_threads > 256) {
            tu = *topology;
            tu.wg_threads = 256;
            topology = &tu;
        }
        bsm_status st = resolve_topology(topology, device, dtype, p->kernel_class, p->shifted,
                                         &p->topo);
        if (st != BSM_OK) return st;
        st = resolve_weights(xcd_weight, &p->topo);
        if (st != BSM_OK) return st;
        p->topo.row_unit = row_unit;
        err = bsm::check_topology(p->topo);
        if (!err.empty()) return fail(BSM_ERR_INVALID_ARG, "topology: %s", err.c_str());
        // planned with one-wave workgroups, so that worker w is workgroup w (on XCD w mod n_xcd)
        bsm::Topology tt = p->topo;
        if (team) tt.wg_threads = 64;
        err = bsm::build_table(p->geo, schedule, tt, home_xcd, p->kernel_class, &p->table);
        if (!err.empty()) return fail(BSM_ERR_INVALID_ARG, "plan: %s", err.c_str());
        if (team) {
            p->table.per_wave = false;
            p->table.stats.per_wave = 0;
            p->table.stats.wg_threads = p->topo.wg_threads;
            p->table.stats.trace_bytes = static_cast<int64_t>(p->topo.n_wg()) *
                                         (p->topo.wg_threads / 64) *
                                         static_cast<int64_t>(sizeof(bsm_trace_rec));
        }
        if (alloc_fail_hook() == AllocFail::host) throw std::bad_alloc();
    } catch (const std::bad_alloc&) {
        return fail(BSM_ERR_OOM, "host allocation failed while planning");
    }
    p->device = device;
    p->dtype = dtype;
    p->schedule = schedule;
    p->flags = topology ? topology->flags : 0;
    p->table.stats.flags = p->flags;
    p->table.stats.dtype = dtype;
    p->table.stats.kernel_class = p->kernel_class;

    if (device >= 0) {
        DeviceGuard g;
        hipError_t e = g.enter(device);
        if (e != hipSuccess) return hip_fail(e, "hipSetDevice");
        if (p->kernel_class >= kLongRowClass) {
            hipDeviceProp_t prop;
            e = hipGetDeviceProperties(&prop, device);
            if (e != hipSuccess) return hip_fail(e, "hipGetDeviceProperties");
            int static_bytes = 0;
            e = bsm::static_lds_bytes(dtype, p->kernel_class, p->shifted, &static_bytes);
            if (e != hipSuccess) return hip_fail(e, "hipFuncGetAttributes");
            const int64_t b = lds_bytes_per_wave(prop, p->topo, static_bytes);
            p->lds_floats_per_wave = static_cast<int>(b / static_cast<int64_t>(sizeof(float)));
            p->table.stats.lds_bytes_per_wave = static_cast<int32_t>(b);
        }
        if (!upload) {
            *out_plan = p.release();
            return BSM_OK;
        }
        const size_t ptr_bytes = p->table.worker_ptr.size() * sizeof(int32_t);
        const size_t items_at = table_items_at(p->table);
        const size_t bytes = table_bytes(p->table);
        e = table_malloc(&p->d_table, bytes);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            p->d_table = nullptr;
            return fail(e == hipErrorOutOfMemory ? BSM_ERR_OOM : BSM_ERR_HIP,
                        "hipMalloc(%zu) for the work table: %s", bytes, hipGetErrorString(e));
        }
        char* base = static_cast<char*>(p->d_table);
        e = hipMemcpy(base, p->table.worker_ptr.data(), ptr_bytes, hipMemcpyHostToDevice);
        if (e == hipSuccess && !p->table.items.empty())
            e = hipMemcpy(base + items_at, p->table.items.data(),
                          p->table.items.size() * sizeof(bsm_item), hipMemcpyHostToDevice);
        if (e != hipSuccess) {
            bsm_status st = hip_fail(e, "uploading the work table");
            free_device(p.get());
            return st;
        }
        p->d_worker_ptr = reinterpret_cast<const int32_t*>(base);
        p->d_items = reinterpret_cast<const bsm_item*>(base + items_at);
    }
    *out_plan = p.release();
    return BSM_OK;
}

// An output may be one of the inputs exactly (in place) or lie apart from it; any other
// overlap of `extent_bytes`-long buffers is refused.
bool partial_overlap(const void* x, const void* y, int64_t extent_bytes) {
    const uintptr_t a = reinterpret_cast<uintptr_t>(x), b = reinterpret_cast<uintptr_t>(y);
    return a != b && a < b + static_cast<uintptr_t>(extent_bytes) &&
           b < a + static_cast<uintptr_t>(extent_bytes);
}

// Forward (b == nullptr: out = softmax(a)) or backward (out = dx of y = a, dy = b).
bsm_status execute_plan(bsm_plan p, bool backward, const void* a, const void* b, void* out,
                        void* stream, void* trace) {
    if (!p) return fail(BSM_ERR_INVALID_ARG, "plan is NULL");
    if (p->gemm) return fail(BSM_ERR_UNSUPPORTED, "a matrix-product plan runs with bsm_gemm_execute");
    if (p->device < 0) return fail(BSM_ERR_UNSUPPORTED, "host-only plan (device -1) cannot execute");
    const int64_t extent_bytes = p->geo.extent * elem_bytes_of(p->dtype);
    if (p->geo.total_elems == 0) return BSM_OK;
    if (!a || !out || (backward && !b)) return fail(BSM_ERR_INVALID_ARG, "an input or the output is NULL");
    if (partial_overlap(a, out, extent_bytes) || (backward && partial_overlap(b, out, extent_bytes)))
        return fail(BSM_ERR_ALIAS, "an input and the output overlap without being equal (extent %lld bytes)",
                    static_cast<long long>(extent_bytes));
    const int es = elem_bytes_of(p->dtype);
    if (reinterpret_cast<uintptr_t>(a) % es != 0 || reinterpret_cast<uintptr_t>(out) % es != 0 ||
        (backward && reinterpret_cast<uintptr_t>(b) % es != 0))
        return fail(BSM_ERR_INVALID_ARG, "a buffer is not aligned to the element size");
    DeviceGuard g;
    hipError_t e = g.enter(p->device);
    if (e != hipSuccess) return hip_fail(e, "hipSetDevice");
    hipStream_t s = static_cast<hipStream_t>(stream);
    const bool temporal = (p->flags & BSM_FLAG_TEMPORAL) != 0;
    if (backward)
        e = bsm::launch_softmax_backward(p->dtype, p->kernel_class, p->shifted, temporal, a, b, out,
                                         p->d_worker_ptr, p->d_items, p->topo.n_wg(),
                                         p->topo.wg_threads, p->table.per_wave ? 1 : 0,
                                         p->lds_floats_per_wave, trace, s);
    else
        e = bsm::launch_softmax(p->dtype, p->kernel_class, p->shifted, temporal, a, out, p->d_worker_ptr,
                                p->d_items, p->topo.n_wg(), p->topo.wg_threads,
                                p->table.per_wave ? 1 : 0, p->lds_floats_per_wave, trace, s);
    if (e != hipSuccess) return hip_fail(e, "kernel launch");
    p->used = true;
    return BSM_OK;
}

// --------------------------------------------------------------------- matrix products
bsm_status create_gemm_plan(bsm_plan* out_plan, int64_t batch, int32_t m, int32_t n, int32_t k,
                            int layout, bsm_dtype out_dtype, bsm_schedule schedule,
                            const int8_t* home_xcd, const bsm_topology* topology, int device,
                            bool upload = true) {
    if (!out_plan) return fail(BSM_ERR_INVALID_ARG, "out_plan is NULL");
    *out_plan = nullptr;
    if (layout != BSM_GEMM_NT && layout != BSM_GEMM_NN && layout != BSM_GEMM_NT_SOFTMAX)
        return fail(BSM_ERR_INVALID_ARG, "unknown layout %d", layout);
    if (batch < 0 || m < 0 || n < 0 || k < 0)
        return fail(BSM_ERR_INVALID_ARG, "negative size (batch %lld, m %d, n %d, k %d)",
                    static_cast<long long>(batch), m, n, k);
    if (static_cast<double>(batch) * std::max({m, n, k}) * std::max({m, n, k}) > 1.0e18)
        return fail(BSM_ERR_INVALID_ARG, "operands too large");
    // The kernel runs workgroups of gemm_wg_threads() threads whose waves share staged operands,
    // gemm_waves_per_simd() per CU by default; each workgroup is one worker of the table.  The
    // score softmax of k <= 128 and 64 < n <= 512 runs in one pass, two workgroups per CU (its
    // LDS does not fit three), unless the topology asks for more.
    bsm_topology t{};
    if (topology) t = *topology;
    const int wg_threads = bsm::gemm_wg_threads();
    if (t.wg_threads != 0 && t.wg_threads != wg_threads)
        return fail(BSM_ERR_INVALID_ARG, "matrix-product plans run %d-thread workgroups (got %d)",
                    wg_threads, t.wg_threads);
    const bool single = layout == BSM_GEMM_NT_SOFTMAX && bsm::gemm_single_pass_shape(n, k) &&
                        (t.wg_per_cu == 0 || t.wg_per_cu <= bsm::gemm_waves_per_simd(true));
    if (t.wg_per_cu == 0) t.wg_per_cu = bsm::gemm_waves_per_simd(single);
    const bool bf16_out = out_dtype == BSM_BF16;
    if (device >= 0) {
        DeviceGuard g;
        hipError_t e = g.enter(device);
        hipDeviceProp_t prop;
        if (e == hipSuccess) e = hipGetDeviceProperties(&prop, device);
        if (e != hipSuccess) return hip_fail(e, "hipGetDeviceProperties");
        const int64_t per_wg = bsm::gemm_lds_bytes_per_wg(bf16_out, single);
        if (per_wg > static_cast<int64_t>(prop.sharedMemPerBlock) ||
            per_wg * t.wg_per_cu > static_cast<int64_t>(prop.maxSharedMemoryPerMultiProcessor))
            return fail(BSM_ERR_INVALID_ARG, "wg_per_cu %d: %lld bytes of LDS per workgroup do not fit",
                        t.wg_per_cu, static_cast<long long>(per_wg));
    }
    // planned with one-wave workgroups, so that every worker is a workgroup (same index, same
    // XCD); the launch then runs the real workgroup size
    t.wg_threads = 64;
    const int32_t rows[1] = {m}, cols[1] = {n};
    bsm_plan p = nullptr;
    bsm_status st = create_plan(&p, nullptr, rows, cols, m == 0 || n == 0 ? 0 : batch, out_dtype,
                                schedule, home_xcd, nullptr, &t, device, bsm::gemm_rows_per_wg(single), true,
                                upload);
    if (st != BSM_OK) return st;
    p->topo.wg_threads = wg_threads;
    p->table.per_wave = false;
    p->table.stats.per_wave = 0;
    p->table.stats.wg_threads = wg_threads;
    p->table.stats.trace_bytes = static_cast<int64_t>(p->topo.n_wg()) * (wg_threads / 64) *
                                 static_cast<int64_t>(sizeof(bsm_trace_rec));
    p->gemm = true;
    p->gemm_m = m;
    p->gemm_n = n;
    p->gemm_k = k;
    p->gemm_layout = layout;
    p->gemm_single = single;
    p->gemm_batch = batch;
    p->table.stats.algorithmic_bytes =
        batch * (2 * (static_cast<int64_t>(m) * k + static_cast<int64_t>(n) * k) +
                 static_cast<int64_t>(m) * n * elem_bytes_of(out_dtype));
    *out_plan = p;
    return BSM_OK;
}

bsm_status execute_gemm(bsm_plan p, const void* a, const void* b, void* c, float alpha,
                        void* stream, void* trace) {
    if (!p) return fail(BSM_ERR_INVALID_ARG, "plan is NULL");
    if (!p->gemm) return fail(BSM_ERR_UNSUPPORTED, "a softmax plan runs with bsm_plan_execute");
    if (p->device < 0) return fail(BSM_ERR_UNSUPPORTED, "host-only plan (device -1) cannot execute");
    const int64_t nb = p->gemm_batch;
    const int64_t a_bytes = nb * p->gemm_m * static_cast<int64_t>(p->gemm_k) * 2;
    const int64_t b_bytes = nb * p->gemm_n * static_cast<int64_t>(p->gemm_k) * 2;
    const int64_t c_bytes = nb * p->gemm_m * static_cast<int64_t>(p->gemm_n) * elem_bytes_of(p->dtype);
    if (c_bytes == 0) return BSM_OK;
    if (!c || !a || !b) return fail(BSM_ERR_INVALID_ARG, "an operand is NULL");
    if (!std::isfinite(alpha)) return fail(BSM_ERR_INVALID_ARG, "alpha must be finite");
    auto overlap = [](const void* x, int64_t xn, const void* y, int64_t yn) {
        const uintptr_t u = reinterpret_cast<uintptr_t>(x), v = reinterpret_cast<uintptr_t>(y);
        return xn > 0 && yn > 0 && u < v + static_cast<uintptr_t>(yn) && v < u + static_cast<uintptr_t>(xn);
    };
    if (overlap(c, c_bytes, a, a_bytes) || overlap(c, c_bytes, b, b_bytes))
        return fail(BSM_ERR_ALIAS, "C overlaps A or B");
    if ((reinterpret_cast<uintptr_t>(a) | reinterpret_cast<uintptr_t>(b)) % 2 != 0 ||
        reinterpret_cast<uintptr_t>(c) % elem_bytes_of(p->dtype) != 0)
        return fail(BSM_ERR_INVALID_ARG, "an operand is not aligned to its element size");
    DeviceGuard g;
    hipError_t e = g.enter(p->device);
    if (e != hipSuccess) return hip_fail(e, "hipSetDevice");
    hipStream_t s = static_cast<hipStream_t>(stream);
    // k == 0 runs the same kernel: an empty reduction stores zeros
    e = bsm::launch_gemm(p->gemm_layout, p->dtype == BSM_BF16, (p->flags & BSM_FLAG_TEMPORAL) != 0,
                         p->gemm_single, a, b, c, p->gemm_m, p->gemm_n,
                         p->gemm_k, alpha, p->d_worker_ptr, p->d_items, p->topo.n_wg(), trace, s);
    if (e != hipSuccess) return hip_fail(e, "kernel launch");
    p->used = true;
    return BSM_OK;
}

// ---------------------------------------------------------------------------- plan cache
// The one-shot calls (bsm_softmax, bsm_softmax_backward, bsm_gemm) run plans from a cache keyed
// by device, op, element type, schedule and the exact geometry.
//
// A hit hashes the caller's geometry arrays, compares them exactly with the stored key and
// launches: no allocation, copy, event or synchronisation, and the launch itself runs outside
// the lock.  A miss builds the plan on the host outside the lock, then uploads its table with
// hipMemcpyAsync on the caller's stream, from a pinned staging buffer into a device buffer,
// both taken from pools that the cache recycles.  Nothing is freed while the cache runs
// (hipFree and hipHostFree synchronise the device): an evicted plan's device buffer goes back
// to the pool tagged with the streams the plan ran on, and whoever takes it next on stream T
// first makes T wait (hipStreamWaitEvent) on an event recorded then on each other tagged
// stream, so the reuse is ordered after every kernel that read the old table while the host
// never waits.  A staging buffer is reused once the event recorded after its copy has
// completed.  A plan that another stream runs before its upload is seen complete makes that
// stream wait on the upload's event.
//
// Graph capture: a hit on a capturing stream pins its plan (never evicted; only
// bsm_cache_clear frees it) once its upload has completed; a miss is refused
// (BSM_ERR_UNSUPPORTED), since building a plan allocates and copies.
constexpr size_t kCacheMax = 32;
constexpr size_t kMaxTrackedStreams = 8;
constexpr size_t kMinPoolBytes = 64 * 1024;

// The caller's geometry, not copied (uniform: R and C have one entry).
struct KeyView {
    int device = 0, kind = 0, dtype = 0, schedule = 0;  // kind 0: softmax, 1: product
    bool uniform = true;
    int64_t batch = 0;
    const int64_t* off = nullptr;
    const int32_t* R = nullptr;
    const int32_t* C = nullptr;
    int32_t gm = 0, gn = 0, gk = 0, glayout = 0;  // products
    int64_t n_entries() const { return uniform ? 1 : batch; }
};

// 64-bit multiply-xorshift over 8-byte words: enough to tell geometries apart before the exact
// comparison.
struct Hasher {
    uint64_t h = 0x9E3779B97F4A7C15ull;
    void word(uint64_t v) {
        h ^= v + 0x9E3779B97F4A7C15ull + (h << 6) + (h >> 2);
        h *= 0xBF58476D1CE4E5B9ull;
        h ^= h >> 31;
    }
    void bytes(const void* p, size_t n) {
        const unsigned char* c = static_cast<const unsigned char*>(p);
        size_t i = 0;
        for (; i + 8 <= n; i += 8) {
            uint64_t v;
            std::memcpy(&v, c + i, 8);
            word(v);
        }
        uint64_t tail = 0;
        std::memcpy(&tail, c + i, n - i);
        word(tail ^ (static_cast<uint64_t>(n) << 56));
    }
};

uint64_t hash_key(const KeyView& k) {
    Hasher h;
    h.word(static_cast<uint64_t>(k.device) | (static_cast<uint64_t>(k.kind) << 16) |
           (static_cast<uint64_t>(k.dtype) << 24) | (static_cast<uint64_t>(k.schedule) << 32) |
           (static_cast<uint64_t>(k.uniform) << 40) | (static_cast<uint64_t>(k.glayout) << 48));
    h.word(static_cast<uint64_t>(k.batch));
    h.word(static_cast<uint64_t>(static_cast<uint32_t>(k.gm)) |
           (static_cast<uint64_t>(static_cast<uint32_t>(k.gn)) << 32));
    h.word(static_cast<uint64_t>(static_cast<uint32_t>(k.gk)));
    const size_t n = static_cast<size_t>(k.n_entries());
    if (k.off) h.bytes(k.off, n * sizeof(int64_t));
    if (k.R) h.bytes(k.R, n * sizeof(int32_t));
    if (k.C) h.bytes(k.C, n * sizeof(int32_t));
    return h.h;
}

struct CacheKey {
    uint64_t hash = 0;
    int device = 0, kind = 0, dtype = 0, schedule = 0;
    bool uniform = true;
    int64_t batch = 0;
    std::vector<int64_t> off;
    std::vector<int32_t> R, C;
    int32_t gm = 0, gn = 0, gk = 0, glayout = 0;
    CacheKey(const KeyView& k, uint64_t h)
        : hash(h), device(k.device), kind(k.kind), dtype(k.dtype), schedule(k.schedule),
          uniform(k.uniform), batch(k.batch), gm(k.gm), gn(k.gn), gk(k.gk), glayout(k.glayout) {
        const size_t n = static_cast<size_t>(k.n_entries());
        if (k.off) off.assign(k.off, k.off + n);
        if (k.R) R.assign(k.R, k.R + n);
        if (k.C) C.assign(k.C, k.C + n);
    }
    bool matches(const KeyView& k, uint64_t h) const {
        if (h != hash || k.device != device || k.kind != kind || k.dtype != dtype ||
            k.schedule != schedule || k.uniform != uniform || k.batch != batch || k.gm != gm ||
            k.gn != gn || k.gk != gk || k.glayout != glayout)
            return false;
        const size_t n = static_cast<size_t>(k.n_entries());
        auto same = [n](const auto& v, const auto* p) {
            if (!p) return v.empty();
            return v.size() == n && (n == 0 || std::memcmp(v.data(), p, n * sizeof(*p)) == 0);
        };
        return same(off, k.off) && same(R, k.R) && same(C, k.C);
    }
};

struct CacheEntry {
    CacheKey key;
    bsm_plan plan;
};

struct DevBuf {  // a device table buffer of the pool
    void* ptr = nullptr;
    size_t bytes = 0;
    std::vector<hipStream_t> after;  // its last reader ran on these streams
};

struct PinBuf {  // a pinned staging buffer of the pool
    void* ptr = nullptr;
    size_t bytes = 0;
    hipEvent_t done = nullptr;  // recorded after the copy that reads it
    bool pending = false;
};

struct DeviceCache {
    std::list<CacheEntry> lru;           // most recently used first
    std::vector<bsm_plan> graveyard;     // evicted, until no call is launching them
    std::vector<DevBuf> free_bufs;       // reusable after stream waits
    std::vector<void*> stale_bufs;       // readers not trackable: freed by bsm_cache_clear only
    std::vector<PinBuf> pins;
};

std::mutex g_cache_mu;
std::vector<std::unique_ptr<DeviceCache>> g_cache;  // by device ordinal

DeviceCache& cache_of(int device) {
    if (static_cast<size_t>(device) >= g_cache.size()) g_cache.resize(device + 1);
    if (!g_cache[device]) g_cache[device].reset(new DeviceCache);
    return *g_cache[device];
}

size_t pool_size(size_t need) {
    size_t b = kMinPoolBytes;
    while (b < need) b *= 2;
    return b;
}

void destroy_plan(bsm_plan p) {
    if (!p) return;
    free_device(p);
    if (p->upload_done) (void)hipEventDestroy(p->upload_done);
    delete p;
}

bool is_capturing(hipStream_t s) {
    hipStreamCaptureStatus st = hipStreamCaptureStatusNone;
    return hipStreamIsCapturing(s, &st) != hipSuccess || st != hipStreamCaptureStatusNone;
}

// Evicted plans no call is launching any more give their buffers back to the pool.
void reclaim(DeviceCache& dc) {
    auto it = dc.graveyard.begin();
    while (it != dc.graveyard.end()) {
        bsm_plan p = *it;
        if (p->inflight.load(std::memory_order_acquire) != 0) {
            ++it;
            continue;
        }
        if (p->d_table) {
            if (p->many_streams)
                dc.stale_bufs.push_back(p->d_table);
            else
                dc.free_bufs.push_back(DevBuf{p->d_table, p->table_cap, p->streams});
        }
        p->d_table = nullptr;
        destroy_plan(p);
        it = dc.graveyard.erase(it);
    }
}

// A device buffer of at least `need` bytes whose reuse is ordered on `stream` after its last
// readers; the stream waits on events recorded on the other streams (no host wait).
bsm_status take_device_buffer(DeviceCache& dc, size_t need, hipStream_t stream, DevBuf* out) {
    reclaim(dc);
    for (;;) {
        int best = -1;
        for (size_t i = 0; i < dc.free_bufs.size(); ++i) {
            const DevBuf& b = dc.free_bufs[i];
            if (b.bytes >= need && b.bytes <= 4 * pool_size(need) &&
                (best < 0 || b.bytes < dc.free_bufs[best].bytes))
                best = static_cast<int>(i);
        }
        if (best < 0) break;
        DevBuf b = dc.free_bufs[best];
        dc.free_bufs.erase(dc.free_bufs.begin() + best);
        bool ok = true;
        for (hipStream_t s : b.after) {
            if (s == stream) continue;
            // a stream that is capturing would take the event into its graph: not now
            if (is_capturing(s)) {
                ok = false;
                break;
            }
            hipEvent_t ev = nullptr;
            if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) != hipSuccess) {
                (void)hipGetLastError();
                ok = false;
                break;
            }
            const bool waited = hipEventRecord(ev, s) == hipSuccess &&
                                hipStreamWaitEvent(stream, ev, 0) == hipSuccess;
            (void)hipEventDestroy(ev);
            if (!waited) {
                (void)hipGetLastError();
                ok = false;
                break;
            }
        }
        if (ok) {
            *out = b;
            return BSM_OK;
        }
        dc.stale_bufs.push_back(b.ptr);
    }
    DevBuf b;
    b.bytes = pool_size(need);
    hipError_t e = table_malloc(&b.ptr, b.bytes);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(e == hipErrorOutOfMemory ? BSM_ERR_OOM : BSM_ERR_HIP,
                    "hipMalloc(%zu) for the work table: %s", b.bytes, hipGetErrorString(e));
    }
    *out = b;
    return BSM_OK;
}

bsm_status take_pinned_buffer(DeviceCache& dc, size_t need, PinBuf** out) {
    PinBuf* best = nullptr;
    for (PinBuf& pb : dc.pins) {
        if (pb.bytes < need || !pb.done) continue;
        if (pb.pending) {
            hipError_t q = hipEventQuery(pb.done);
            if (q == hipErrorNotReady) {
                (void)hipGetLastError();  // not an error: leave no state behind for the caller
                continue;
            }
            if (q != hipSuccess) return hip_fail(q, "hipEventQuery");
            pb.pending = false;
        }
        if (!best || pb.bytes < best->bytes) best = &pb;
    }
    if (!best) {
        PinBuf pb;
        pb.bytes = pool_size(need);
        hipError_t e = hipHostMalloc(&pb.ptr, pb.bytes, hipHostMallocDefault);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            return fail(e == hipErrorOutOfMemory ? BSM_ERR_OOM : BSM_ERR_HIP,
                        "hipHostMalloc(%zu) for table staging: %s", pb.bytes, hipGetErrorString(e));
        }
        e = hipEventCreateWithFlags(&pb.done, hipEventDisableTiming);
        if (e != hipSuccess) {
            dc.pins.push_back(pb);  // the buffer is kept (freeing it would synchronise)
            dc.pins.back().done = nullptr;
            return hip_fail(e, "hipEventCreateWithFlags");
        }
        dc.pins.push_back(pb);
        best = &dc.pins.back();
    }
    *out = best;
    return BSM_OK;
}

// Uploads a freshly built plan's table on `stream` (caller holds the lock).
bsm_status upload_pooled(DeviceCache& dc, bsm_plan p, hipStream_t stream) {
    const size_t need = table_bytes(p->table);
    const size_t items_at = table_items_at(p->table);
    DevBuf buf;
    bsm_status st = take_device_buffer(dc, need, stream, &buf);
    if (st != BSM_OK) return st;
    PinBuf* pin = nullptr;
    st = take_pinned_buffer(dc, need, &pin);
    if (st != BSM_OK || !pin->done) {
        dc.free_bufs.push_back(DevBuf{buf.ptr, buf.bytes, {stream}});
        return st != BSM_OK ? st : fail(BSM_ERR_HIP, "no staging event");
    }
    char* h = static_cast<char*>(pin->ptr);
    std::memcpy(h, p->table.worker_ptr.data(), p->table.worker_ptr.size() * sizeof(int32_t));
    if (!p->table.items.empty())
        std::memcpy(h + items_at, p->table.items.data(), p->table.items.size() * sizeof(bsm_item));
    hipEvent_t up = nullptr;
    hipError_t e = hipEventCreateWithFlags(&up, hipEventDisableTiming);
    if (e == hipSuccess) e = hipMemcpyAsync(buf.ptr, h, need, hipMemcpyHostToDevice, stream);
    if (e == hipSuccess) e = hipEventRecord(pin->done, stream);
    if (e == hipSuccess) {
        pin->pending = true;
        e = hipEventRecord(up, stream);
    }
    if (e != hipSuccess) {
        if (up) (void)hipEventDestroy(up);
        dc.free_bufs.push_back(DevBuf{buf.ptr, buf.bytes, {stream}});
        return hip_fail(e, "uploading the work table");
    }
    p->pooled = true;
    p->d_table = buf.ptr;
    p->table_cap = buf.bytes;
    p->d_worker_ptr = static_cast<const int32_t*>(buf.ptr);
    p->d_items = reinterpret_cast<const bsm_item*>(static_cast<char*>(buf.ptr) + items_at);
    p->upload_stream = stream;
    p->upload_done = up;
    p->uploaded = false;
    return BSM_OK;
}

// Hit bookkeeping (caller holds the lock): order the call after the table upload, track the
// stream, pin a captured plan.
bsm_status prepare_call(bsm_plan p, hipStream_t stream, bool capturing) {
    if (!p->uploaded) {
        hipError_t q = p->upload_done ? hipEventQuery(p->upload_done) : hipSuccess;
        if (q == hipSuccess) {
            p->uploaded = true;
        } else if (capturing) {
            (void)hipGetLastError();
            return fail(BSM_ERR_UNSUPPORTED,
                        "one-shot call under stream capture while its plan's table upload is "
                        "still in flight; synchronise once before capturing");
        } else if (q == hipErrorNotReady) {
            (void)hipGetLastError();  // not an error: leave no state behind for the caller
            if (stream != p->upload_stream) {
                hipError_t e = hipStreamWaitEvent(stream, p->upload_done, 0);
                if (e != hipSuccess) return hip_fail(e, "hipStreamWaitEvent");
            }
        } else {
            return hip_fail(q, "hipEventQuery");
        }
    }
    if (std::find(p->streams.begin(), p->streams.end(), stream) == p->streams.end()) {
        if (p->streams.size() < kMaxTrackedStreams)
            p->streams.push_back(stream);
        else
            p->many_streams = true;
    }
    if (capturing) p->captured = true;
    p->inflight.fetch_add(1, std::memory_order_acq_rel);
    return BSM_OK;
}

bsm_plan lookup(DeviceCache& dc, const KeyView& kv, uint64_t h) {
    for (auto it = dc.lru.begin(); it != dc.lru.end(); ++it) {
        if (it->key.matches(kv, h)) {
            if (it != dc.lru.begin()) dc.lru.splice(dc.lru.begin(), dc.lru, it);
            return dc.lru.front().plan;
        }
    }
    return nullptr;
}

void evict(DeviceCache& dc) {
    auto it = dc.lru.end();
    while (dc.lru.size() > kCacheMax && it != dc.lru.begin()) {
        --it;
        if (it->plan->captured) continue;
        dc.graveyard.push_back(it->plan);
        it = dc.lru.erase(it);
    }
}

// Runs `launch(plan)` on the cached plan for `kv`, building it with `build(&plan)` (a plan
// with its table on the host only) on a miss.
template <class Build, class Launch>
bsm_status run_cached(const KeyView& kv, hipStream_t stream, Build build, Launch launch) {
    const uint64_t h = hash_key(kv);
    const bool capturing = is_capturing(stream);
    bsm_plan plan = nullptr;
    {
        std::lock_guard<std::mutex> lock(g_cache_mu);
        DeviceCache& dc = cache_of(kv.device);
        plan = lookup(dc, kv, h);
        if (plan) {
            bsm_status st = prepare_call(plan, stream, capturing);
            if (st != BSM_OK) return st;
        }
    }
    if (!plan) {
        if (capturing)
            return fail(BSM_ERR_UNSUPPORTED,
                        "one-shot call under stream capture with a geometry not in the plan cache "
                        "(building a plan allocates and copies); run it once before capturing, "
                        "or capture a plan's execution");
        bsm_plan fresh = nullptr;
        bsm_status st = build(&fresh);
        if (st != BSM_OK) return st;
        std::unique_ptr<bsm_plan_s> owner(fresh);  // no device memory yet
        DeviceGuard g;
        hipError_t e = g.enter(kv.device);
        if (e != hipSuccess) return hip_fail(e, "hipSetDevice");
        std::lock_guard<std::mutex> lock(g_cache_mu);
        DeviceCache& dc = cache_of(kv.device);
        plan = lookup(dc, kv, h);  // another thread may have built it meanwhile
        if (!plan) {
            try {
                dc.lru.push_front(CacheEntry{CacheKey(kv, h), fresh});
            } catch (const std::bad_alloc&) {
                return fail(BSM_ERR_OOM, "host allocation failed (plan cache)");
            }
            st = upload_pooled(dc, fresh, stream);
            if (st != BSM_OK) {
                dc.lru.pop_front();
                return st;
            }
            plan = owner.release();
            evict(dc);
        }
        st = prepare_call(plan, stream, false);
        if (st != BSM_OK) return st;
    }
    bsm_status st = launch(plan);
    plan->inflight.fetch_sub(1, std::memory_order_acq_rel);
    return st;
}

// Argument checks of the one-shot calls, before any HIP call (allocation-free in the common
// case of slices in ascending order).  *extent = 0: nothing to do.
bsm_status check_one_shot(bool backward, const void* a, const void* b, const void* out,
                          const int64_t* slice_offsets, const int32_t* rows, const int32_t* cols,
                          int64_t batch, bsm_dtype dtype, bsm_schedule schedule, int64_t* extent_out) {
    *extent_out = 0;
    if (!valid_dtype(dtype)) return fail(BSM_ERR_INVALID_ARG, "unknown dtype %d", static_cast<int>(dtype));
    if (!valid_schedule(schedule)) return fail(BSM_ERR_INVALID_ARG, "unknown schedule %d", static_cast<int>(schedule));
    int64_t extent = 0;
    if (!bsm::quick_geometry(slice_offsets, rows, cols, batch, &extent)) {
        bsm::Geometry geo;
        std::string err;
        try {
            err = bsm::make_geometry(slice_offsets, rows, cols, batch, elem_bytes_of(dtype), &geo);
        } catch (const std::bad_alloc&) {
            return fail(BSM_ERR_OOM, "host allocation failed");
        }
        if (!err.empty()) return fail(BSM_ERR_INVALID_ARG, "geometry: %s", err.c_str());
        extent = geo.extent;
    }
    if (extent == 0) return BSM_OK;  // no element: nothing to do
    if (!a || !out || (backward && !b)) return fail(BSM_ERR_INVALID_ARG, "an input or the output is NULL");
    const int64_t extent_bytes = extent * elem_bytes_of(dtype);
    if (partial_overlap(a, out, extent_bytes) || (backward && partial_overlap(b, out, extent_bytes)))
        return fail(BSM_ERR_ALIAS, "an input and the output overlap without being equal");
    *extent_out = extent;
    return BSM_OK;
}

// One-shot call: checked arguments, then a cached plan for the geometry runs.
bsm_status one_shot(bool backward, const void* a, const void* b, void* out,
                    const int64_t* slice_offsets, const int32_t* rows, const int32_t* cols,
                    int64_t batch, bsm_dtype dtype, bsm_schedule schedule, void* stream) {
    int64_t extent = 0;
    bsm_status st = check_one_shot(backward, a, b, out, slice_offsets, rows, cols, batch, dtype,
                                   schedule, &extent);
    if (st != BSM_OK || extent == 0) return st;
    int device = 0;
    hipError_t e = hipGetDevice(&device);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    KeyView kv;
    kv.device = device;
    kv.kind = 0;
    kv.dtype = dtype;
    kv.schedule = schedule;
    kv.uniform = slice_offsets == nullptr;
    kv.batch = batch;
    kv.off = slice_offsets;
    kv.R = rows;
    kv.C = cols;
    return run_cached(
        kv, static_cast<hipStream_t>(stream),
        [&](bsm_plan* np) {
            return create_plan(np, slice_offsets, rows, cols, batch, dtype, schedule, nullptr,
                               nullptr, nullptr, device, 0, false, false);
        },
        [&](bsm_plan p) { return execute_plan(p, backward, a, b, out, stream, nullptr); });
}

// bsm_softmax with the work table in the library's static device buffer: the plan is built on
// the host for this call only and its table copied into the buffer on `stream`; nothing is
// allocated on the device or pinned.
bsm_status softmax_noalloc(const void* in, void* out, const int64_t* slice_offsets,
                           const int32_t* rows, const int32_t* cols, int64_t batch,
                           bsm_dtype dtype, bsm_schedule schedule, void* stream) {
    int64_t extent = 0;
    bsm_status st = check_one_shot(false, in, nullptr, out, slice_offsets, rows, cols, batch,
                                   dtype, schedule, &extent);
    if (st != BSM_OK || extent == 0) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (is_capturing(s))
        return fail(BSM_ERR_UNSUPPORTED, "bsm_softmax_noalloc under stream capture (its table "
                                         "copy waits for the stream)");
    int device = 0;
    hipError_t e = hipGetDevice(&device);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    bsm_plan raw = nullptr;
    st = create_plan(&raw, slice_offsets, rows, cols, batch, dtype, schedule, nullptr, nullptr,
                     nullptr, device, 0, false, false);
    if (st != BSM_OK) return st;
    std::unique_ptr<bsm_plan_s> p(raw);  // host table only
    const size_t need = table_bytes(p->table);
    if (need > static_cast<size_t>(BSM_NOALLOC_SCRATCH_BYTES))
        return fail(BSM_ERR_INVALID_ARG,
                    "work table of %zu bytes (%lld items) exceeds the %d bytes of the "
                    "bsm_softmax_noalloc buffer",
                    need, static_cast<long long>(p->table.items.size()), BSM_NOALLOC_SCRATCH_BYTES);
    void* scratch_ptr = nullptr;
    e = bsm::noalloc_scratch(device, &scratch_ptr);
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress of the static buffer");
    char* base = static_cast<char*>(scratch_ptr);
    const size_t items_at = table_items_at(p->table);
    // pageable sources: the copies complete before they return, in stream order on `s`
    e = hipMemcpyAsync(base, p->table.worker_ptr.data(),
                       p->table.worker_ptr.size() * sizeof(int32_t), hipMemcpyHostToDevice, s);
    if (e == hipSuccess && !p->table.items.empty())
        e = hipMemcpyAsync(base + items_at, p->table.items.data(),
                           p->table.items.size() * sizeof(bsm_item), hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);  // the host table is freed on return
    if (e != hipSuccess) return hip_fail(e, "copying the work table to the static buffer");
    p->pooled = true;  // the buffer is not the plan's
    p->d_worker_ptr = reinterpret_cast<const int32_t*>(base);
    p->d_items = reinterpret_cast<const bsm_item*>(base + items_at);
    return execute_plan(p.get(), false, in, nullptr, out, stream, nullptr);
}

}  // namespace

extern "C" {

bsm_status bsm_plan_create(bsm_plan* out_plan, const int64_t* slice_offsets, const int32_t* rows,
                           const int32_t* cols, int64_t batch, bsm_dtype dtype,
                           bsm_schedule schedule, const int8_t* home_xcd,
                           const bsm_topology* topology, int device) {
    return create_plan(out_plan, slice_offsets, rows, cols, batch, dtype, schedule, home_xcd,
                       nullptr, topology, device);
}

bsm_status bsm_plan_create_weighted(bsm_plan* out_plan, const int64_t* slice_offsets,
                                    const int32_t* rows, const int32_t* cols, int64_t batch,
                                    bsm_dtype dtype, bsm_schedule schedule,
                                    const int8_t* home_xcd, const float* xcd_weight,
                                    const bsm_topology* topology, int device) {
    return create_plan(out_plan, slice_offsets, rows, cols, batch, dtype, schedule, home_xcd,
                       xcd_weight, topology, device);
}

bsm_status bsm_plan_execute(bsm_plan plan, const void* in, void* out, void* stream, void* trace) {
    return execute_plan(plan, false, in, nullptr, out, stream, trace);
}

bsm_status bsm_plan_execute_backward(bsm_plan plan, const void* y, const void* dy, void* dx,
                                     void* stream, void* trace) {
    return execute_plan(plan, true, y, dy, dx, stream, trace);
}

bsm_status bsm_plan_describe(bsm_plan plan, bsm_plan_stats* stats) {
    if (!plan || !stats) return fail(BSM_ERR_INVALID_ARG, "plan or stats is NULL");
    *stats = plan->table.stats;
    return BSM_OK;
}

bsm_status bsm_plan_export(bsm_plan plan, int32_t* worker_ptr, bsm_item* items, int8_t* home,
                           uint8_t* overlap) {
    if (!plan) return fail(BSM_ERR_INVALID_ARG, "plan is NULL");
    const bsm::Table& t = plan->table;
    if (worker_ptr) std::memcpy(worker_ptr, t.worker_ptr.data(), t.worker_ptr.size() * sizeof(int32_t));
    if (items && !t.items.empty()) std::memcpy(items, t.items.data(), t.items.size() * sizeof(bsm_item));
    if (home && !t.home.empty()) std::memcpy(home, t.home.data(), t.home.size());
    if (overlap && !t.overlap.empty()) std::memcpy(overlap, t.overlap.data(), t.overlap.size());
    return BSM_OK;
}

bsm_status bsm_plan_destroy(bsm_plan plan) {
    if (!plan) return fail(BSM_ERR_INVALID_ARG, "plan is NULL");
    destroy_plan(plan);
    return BSM_OK;
}

bsm_status bsm_softmax(const void* in, void* out, const int64_t* slice_offsets, const int32_t* rows,
                       const int32_t* cols, int64_t batch, bsm_dtype dtype, bsm_schedule schedule,
                       void* stream) {
    return one_shot(false, in, nullptr, out, slice_offsets, rows, cols, batch, dtype, schedule,
                    stream);
}

bsm_status bsm_softmax_noalloc(const void* in, void* out, const int64_t* slice_offsets,
                               const int32_t* rows, const int32_t* cols, int64_t batch,
                               bsm_dtype dtype, bsm_schedule schedule, void* stream) {
    return softmax_noalloc(in, out, slice_offsets, rows, cols, batch, dtype, schedule, stream);
}

bsm_status bsm_gemm_plan_create(bsm_plan* out_plan, int64_t batch, int32_t m, int32_t n,
                                int32_t k, bsm_gemm_layout layout, bsm_dtype out_dtype,
                                bsm_schedule schedule, const int8_t* home_xcd,
                                const bsm_topology* topology, int device) {
    return create_gemm_plan(out_plan, batch, m, n, k, static_cast<int>(layout), out_dtype, schedule,
                            home_xcd, topology, device);
}

bsm_status bsm_gemm_execute(bsm_plan plan, const void* a, const void* b, void* c, float alpha,
                            void* stream, void* trace) {
    return execute_gemm(plan, a, b, c, alpha, stream, trace);
}

bsm_status bsm_gemm(const void* a, const void* b, void* c, int64_t batch, int32_t m, int32_t n,
                    int32_t k, bsm_gemm_layout layout, bsm_dtype out_dtype, float alpha,
                    bsm_schedule schedule, void* stream) {
    if (!valid_dtype(out_dtype)) return fail(BSM_ERR_INVALID_ARG, "unknown dtype %d", static_cast<int>(out_dtype));
    if (!valid_schedule(schedule)) return fail(BSM_ERR_INVALID_ARG, "unknown schedule %d", static_cast<int>(schedule));
    if (layout != BSM_GEMM_NT && layout != BSM_GEMM_NN && layout != BSM_GEMM_NT_SOFTMAX)
        return fail(BSM_ERR_INVALID_ARG, "unknown layout %d", static_cast<int>(layout));
    if (batch < 0 || m < 0 || n < 0 || k < 0) return fail(BSM_ERR_INVALID_ARG, "negative size");
    if (batch == 0 || m == 0 || n == 0) return BSM_OK;
    if (!a || !b || !c) return fail(BSM_ERR_INVALID_ARG, "an operand is NULL");
    int device = 0;
    hipError_t e = hipGetDevice(&device);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    KeyView kv;
    kv.device = device;
    kv.kind = 1;
    kv.dtype = out_dtype;
    kv.schedule = schedule;
    kv.batch = batch;
    kv.gm = m;
    kv.gn = n;
    kv.gk = k;
    kv.glayout = static_cast<int>(layout);
    return run_cached(
        kv, static_cast<hipStream_t>(stream),
        [&](bsm_plan* np) {
            return create_gemm_plan(np, batch, m, n, k, static_cast<int>(layout), out_dtype,
                                    schedule, nullptr, nullptr, device, false);
        },
        [&](bsm_plan p) { return execute_gemm(p, a, b, c, alpha, stream, nullptr); });
}

bsm_status bsm_softmax_backward(const void* y, const void* dy, void* dx,
                                const int64_t* slice_offsets, const int32_t* rows,
                                const int32_t* cols, int64_t batch, bsm_dtype dtype,
                                bsm_schedule schedule, void* stream) {
    return one_shot(true, y, dy, dx, slice_offsets, rows, cols, batch, dtype, schedule, stream);
}

bsm_status bsm_cache_clear(void) {
    std::lock_guard<std::mutex> lock(g_cache_mu);
    for (size_t d = 0; d < g_cache.size(); ++d) {
        if (!g_cache[d]) continue;
        DeviceCache& dc = *g_cache[d];
        // calls that found their plan before the lock was taken finish their launch first
        for (bool busy = true; busy;) {
            busy = false;
            for (auto& ent : dc.lru) busy = busy || ent.plan->inflight.load() != 0;
            for (bsm_plan p : dc.graveyard) busy = busy || p->inflight.load() != 0;
            if (busy) std::this_thread::yield();
        }
        DeviceGuard g;
        if (g.enter(static_cast<int>(d)) == hipSuccess) (void)hipDeviceSynchronize();
        for (auto& ent : dc.lru) dc.graveyard.push_back(ent.plan);
        dc.lru.clear();
        reclaim(dc);
        for (DevBuf& b : dc.free_bufs) (void)hipFree(b.ptr);
        for (void* ptr : dc.stale_bufs) (void)hipFree(ptr);
        for (PinBuf& pb : dc.pins) {
            (void)hipHostFree(pb.ptr);
            if (pb.done) (void)hipEventDestroy(pb.done);
        }
        g_cache[d].reset();
    }
    return BSM_OK;
}

bsm_status bsm_device_info(int device, bsm_device_props* info) {
    if (!info) return fail(BSM_ERR_INVALID_ARG, "info is NULL");
    hipDeviceProp_t prop;
    hipError_t e = hipGetDeviceProperties(&prop, device);
    if (e != hipSuccess) return hip_fail(e, "hipGetDeviceProperties");
    std::memset(info, 0, sizeof *info);
    int n_xcd = 1;
    if (hipDeviceGetAttribute(&n_xcd, hipDeviceAttributeNumberOfXccs, device) != hipSuccess) n_xcd = 1;
    int wall = 0;
    if (hipDeviceGetAttribute(&wall, hipDeviceAttributeWallClockRate, device) != hipSuccess) wall = 0;
    info->n_cu = prop.multiProcessorCount;
    info->n_xcd = n_xcd;
    info->wave_size = prop.warpSize;
    info->max_threads_per_cu = prop.maxThreadsPerMultiProcessor;
    info->lds_bytes_per_cu = static_cast<int64_t>(prop.maxSharedMemoryPerMultiProcessor);
    info->lds_bytes_per_wg = static_cast<int64_t>(prop.sharedMemPerBlock);
    info->l2_bytes = prop.l2CacheSize;
    info->hbm_bytes = static_cast<int64_t>(prop.totalGlobalMem);
    info->wall_clock_hz = static_cast<int64_t>(wall) * 1000;  // attribute is in kHz
    info->clock_khz = prop.clockRate;
    info->peak_hbm_gbs = 2.0 * static_cast<double>(prop.memoryClockRate) * 1e3 *
                         (static_cast<double>(prop.memoryBusWidth) / 8.0) / 1e9;
    std::snprintf(info->arch, sizeof info->arch, "%s", prop.gcnArchName);
    return BSM_OK;
}

bsm_status bsm_default_topology(int device, bsm_topology* topology) {
    if (!topology) return fail(BSM_ERR_INVALID_ARG, "topology is NULL");
    return default_topology(device, topology);
}

bsm_status bsm_copy(const void* src, void* dst, int64_t bytes, void* stream) {
    if (bytes < 0) return fail(BSM_ERR_INVALID_ARG, "bytes is negative");
    if (bytes == 0) return BSM_OK;
    if (!src || !dst) return fail(BSM_ERR_INVALID_ARG, "src or dst is NULL");
    const uintptr_t a = reinterpret_cast<uintptr_t>(src), b = reinterpret_cast<uintptr_t>(dst);
    if (a < b + static_cast<uintptr_t>(bytes) && b < a + static_cast<uintptr_t>(bytes))
        return fail(BSM_ERR_ALIAS, "src and dst overlap");
    int device = 0, n_cu = 256;
    if (hipGetDevice(&device) == hipSuccess)
        (void)hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, device);
    hipError_t e = bsm::launch_copy(src, dst, bytes, n_cu, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "copy kernel launch");
    return BSM_OK;
}

const char* bsm_status_string(bsm_status status) {
    switch (status) {
        case BSM_OK: return "BSM_OK";
        case BSM_ERR_INVALID_ARG: return "BSM_ERR_INVALID_ARG";
        case BSM_ERR_UNSUPPORTED: return "BSM_ERR_UNSUPPORTED";
        case BSM_ERR_ALIAS: return "BSM_ERR_ALIAS";
        case BSM_ERR_OOM: return "BSM_ERR_OOM";
        case BSM_ERR_HIP: return "BSM_ERR_HIP";
        default: break;  // any other value, BSM_STATUS_MAX_ENUM included
    }
    return "BSM_ERR_UNKNOWN";
}

const char* bsm_last_error(void) { return g_error.c_str(); }

int32_t bsm_abi_version(void) { return BSM_ABI_VERSION; }

}  // extern "C"
