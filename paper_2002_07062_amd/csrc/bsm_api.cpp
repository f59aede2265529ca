// C-ABI of libbsm.so: argument checks, plans (host table + device copy), the one-shot plan
// cache, device queries and the copy reference.  Every failure is a status code plus a
// thread-local message; nothing is thrown across the ABI.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <list>
#include <memory>
#include <mutex>
#include <new>
#include <string>
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
    // the outputs C_b (gemm_m x gemm_n), A_b is gemm_m x gemm_k, layout 0 = NT, 1 = NN.
    bool gemm = false;
    int gemm_m = 0, gemm_n = 0, gemm_k = 0, gemm_layout = 0;
    int64_t gemm_batch = 0;
    int lds_floats_per_wave = 0;  // one-wave long-row staging (kernel classes 4, 5 on a device)
    int32_t flags = 0;            // BSM_FLAG_* bits
    void* d_table = nullptr;  // device copy: worker_ptr, then items (256-byte aligned)
    const int32_t* d_worker_ptr = nullptr;
    const bsm_item* d_items = nullptr;
    std::atomic<bool> used{false};  // executed at least once (destroy then waits for the device)
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
    if (p->device < 0) return;
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

bsm_status create_plan(bsm_plan* out_plan, const int64_t* offs, const int32_t* rows,
                       const int32_t* cols, int64_t batch, bsm_dtype dtype, bsm_schedule schedule,
                       const int8_t* home_xcd, const float* xcd_weight,
                       const bsm_topology* topology, int device, int32_t row_unit = 0,
                       bool product = false) {
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
        const size_t ptr_bytes = p->table.worker_ptr.size() * sizeof(int32_t);
        const size_t items_at = (ptr_bytes + 255) & ~static_cast<size_t>(255);
        const size_t bytes = items_at + std::max<size_t>(p->table.items.size(), 1) * sizeof(bsm_item);
        e = hipMalloc(&p->d_table, bytes);
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
                            const int8_t* home_xcd, const bsm_topology* topology, int device) {
    if (!out_plan) return fail(BSM_ERR_INVALID_ARG, "out_plan is NULL");
    *out_plan = nullptr;
    if (layout != 0 && layout != 1) return fail(BSM_ERR_INVALID_ARG, "unknown layout %d", layout);
    if (batch < 0 || m < 0 || n < 0 || k < 0)
        return fail(BSM_ERR_INVALID_ARG, "negative size (batch %lld, m %d, n %d, k %d)",
                    static_cast<long long>(batch), m, n, k);
    if (static_cast<double>(batch) * std::max({m, n, k}) * std::max({m, n, k}) > 1.0e18)
        return fail(BSM_ERR_INVALID_ARG, "operands too large");
    // The kernel runs workgroups of gemm_wg_threads() threads whose waves share staged operands,
    // gemm_waves_per_simd() per CU by default; each workgroup is one worker of the table.
    bsm_topology t{};
    if (topology) t = *topology;
    const int wg_threads = bsm::gemm_wg_threads();
    if (t.wg_threads != 0 && t.wg_threads != wg_threads)
        return fail(BSM_ERR_INVALID_ARG, "matrix-product plans run %d-thread workgroups (got %d)",
                    wg_threads, t.wg_threads);
    if (t.wg_per_cu == 0) t.wg_per_cu = bsm::gemm_waves_per_simd();
    const bool bf16_out = out_dtype == BSM_BF16;
    if (device >= 0) {
        DeviceGuard g;
        hipError_t e = g.enter(device);
        hipDeviceProp_t prop;
        if (e == hipSuccess) e = hipGetDeviceProperties(&prop, device);
        if (e != hipSuccess) return hip_fail(e, "hipGetDeviceProperties");
        const int64_t per_wg = bsm::gemm_lds_bytes_per_wg(bf16_out);
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
                                schedule, home_xcd, nullptr, &t, device, bsm::gemm_rows_per_wg(), true);
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
                         a, b, c, p->gemm_m, p->gemm_n,
                         p->gemm_k, alpha, p->d_worker_ptr, p->d_items, p->topo.n_wg(), trace, s);
    if (e != hipSuccess) return hip_fail(e, "kernel launch");
    p->used = true;
    return BSM_OK;
}

// ---------------------------------------------------------------------------- plan cache
struct CacheKey {
    int device;
    int dtype;
    int schedule;
    bool uniform;
    int64_t batch;
    std::vector<int64_t> off;
    std::vector<int32_t> R, C;
    int gemm_k = -1;  // >= 0: a matrix-product plan with this reduction depth
    int gemm_layout = 0;
    bool operator==(const CacheKey& o) const {
        return device == o.device && dtype == o.dtype && schedule == o.schedule &&
               uniform == o.uniform && batch == o.batch && off == o.off && R == o.R && C == o.C &&
               gemm_k == o.gemm_k && gemm_layout == o.gemm_layout;
    }
};

// Looks up (or builds and inserts) the cached plan for `key`; the caller holds g_cache_mu.
template <class Build>
bsm_status cached_plan(CacheKey key, Build build, bsm_plan* out);

struct CacheEntry {
    CacheKey key;
    bsm_plan plan;
};

std::mutex g_cache_mu;
std::list<CacheEntry> g_cache;  // most recently used first
constexpr size_t kCacheMax = 32;

void destroy_plan(bsm_plan p) {
    if (!p) return;
    free_device(p);
    delete p;
}

template <class Build>
bsm_status cached_plan(CacheKey key, Build build, bsm_plan* out) {
    for (auto it = g_cache.begin(); it != g_cache.end(); ++it) {
        if (it->key == key) {
            *out = it->plan;
            g_cache.splice(g_cache.begin(), g_cache, it);
            return BSM_OK;
        }
    }
    bsm_plan plan = nullptr;
    bsm_status st = build(&plan);
    if (st != BSM_OK) return st;
    g_cache.push_front(CacheEntry{std::move(key), plan});
    while (g_cache.size() > kCacheMax) {
        destroy_plan(g_cache.back().plan);
        g_cache.pop_back();
    }
    *out = plan;
    return BSM_OK;
}

// One-shot call: validates the geometry (no HIP call for bad arguments or no-ops), then runs a
// plan from the per-device cache (built on a miss; plans do not depend on the op).
bsm_status one_shot(bool backward, const void* a, const void* b, void* out,
                    const int64_t* slice_offsets, const int32_t* rows, const int32_t* cols,
                    int64_t batch, bsm_dtype dtype, bsm_schedule schedule, void* stream) {
    if (!valid_dtype(dtype)) return fail(BSM_ERR_INVALID_ARG, "unknown dtype %d", static_cast<int>(dtype));
    if (!valid_schedule(schedule)) return fail(BSM_ERR_INVALID_ARG, "unknown schedule %d", static_cast<int>(schedule));
    bsm::Geometry geo;
    std::string err;
    try {
        err = bsm::make_geometry(slice_offsets, rows, cols, batch, elem_bytes_of(dtype), &geo);
    } catch (const std::bad_alloc&) {
        return fail(BSM_ERR_OOM, "host allocation failed");
    }
    if (!err.empty()) return fail(BSM_ERR_INVALID_ARG, "geometry: %s", err.c_str());
    if (geo.total_elems == 0) return BSM_OK;
    if (!a || !out || (backward && !b)) return fail(BSM_ERR_INVALID_ARG, "an input or the output is NULL");
    const int64_t extent_bytes = geo.extent * elem_bytes_of(dtype);
    if (partial_overlap(a, out, extent_bytes) || (backward && partial_overlap(b, out, extent_bytes)))
        return fail(BSM_ERR_ALIAS, "an input and the output overlap without being equal");

    int device = 0;
    hipError_t e = hipGetDevice(&device);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    CacheKey key{device, dtype, schedule, slice_offsets == nullptr, batch, {}, {}, {}};
    if (slice_offsets) {
        key.off.assign(slice_offsets, slice_offsets + batch);
        key.R.assign(rows, rows + batch);
        key.C.assign(cols, cols + batch);
    } else {
        key.R.assign(rows, rows + 1);
        key.C.assign(cols, cols + 1);
    }
    std::lock_guard<std::mutex> lock(g_cache_mu);
    bsm_plan plan = nullptr;
    bsm_status st = cached_plan(std::move(key), [&](bsm_plan* np) {
        return create_plan(np, slice_offsets, rows, cols, batch, dtype, schedule, nullptr, nullptr,
                           nullptr, device);
    }, &plan);
    if (st != BSM_OK) return st;
    return execute_plan(plan, backward, a, b, out, stream, nullptr);
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
    if (layout != BSM_GEMM_NT && layout != BSM_GEMM_NN)
        return fail(BSM_ERR_INVALID_ARG, "unknown layout %d", static_cast<int>(layout));
    if (batch < 0 || m < 0 || n < 0 || k < 0) return fail(BSM_ERR_INVALID_ARG, "negative size");
    if (batch == 0 || m == 0 || n == 0) return BSM_OK;
    if (!a || !b || !c) return fail(BSM_ERR_INVALID_ARG, "an operand is NULL");
    int device = 0;
    hipError_t e = hipGetDevice(&device);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    CacheKey key{device, out_dtype, schedule, true, batch, {}, {m}, {n}, k, static_cast<int>(layout)};
    std::lock_guard<std::mutex> lock(g_cache_mu);
    bsm_plan plan = nullptr;
    bsm_status st = cached_plan(std::move(key), [&](bsm_plan* np) {
        return create_gemm_plan(np, batch, m, n, k, static_cast<int>(layout), out_dtype, schedule,
                                nullptr, nullptr, device);
    }, &plan);
    if (st != BSM_OK) return st;
    return execute_gemm(plan, a, b, c, alpha, stream, nullptr);
}

bsm_status bsm_softmax_backward(const void* y, const void* dy, void* dx,
                                const int64_t* slice_offsets, const int32_t* rows,
                                const int32_t* cols, int64_t batch, bsm_dtype dtype,
                                bsm_schedule schedule, void* stream) {
    return one_shot(true, y, dy, dx, slice_offsets, rows, cols, batch, dtype, schedule, stream);
}

bsm_status bsm_cache_clear(void) {
    std::lock_guard<std::mutex> lock(g_cache_mu);
    for (auto& ent : g_cache) destroy_plan(ent.plan);
    g_cache.clear();
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
