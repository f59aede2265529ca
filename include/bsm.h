/*
 * bsm.h -- batched row softmax over packed 2-D slices, with slice-to-workgroup scheduling,
 *          for AMD Instinct MI355X (gfx950).  Plain C ABI of libbsm.so.
 *
 * The operation (the paper's problem statement, Section 2): B small slices, slice s being an
 * R_s x C_s row-major matrix, are packed into one buffer (for BERT, 384 attention-score slices
 * of 512 x 512 stacked along rows as a 196608 x 512 tensor).  Softmax runs on every row of
 * every slice:
 *
 *     y[s][r][j] = exp(x[s][r][j] - m) / sum_k exp(x[s][r][k] - m),   m = max_k x[s][r][k]
 *
 * and the library decides which persistent workgroup processes which rows (Sections 3 to 5 of
 * the paper: round-robin batch-to-core scheduling as the prior solution; cluster beamforming
 * plus load balancing, with a MINIMAX objective, as the proposed one).  On MI355X a
 * "cluster/core" is a persistent workgroup and a "memory bank" is an XCD with its own L2.
 *
 * Common conventions
 *   - Ownership: the caller owns every input, output and metadata buffer; the library owns
 *     plans, the plan cache and the device copies of work tables.
 *   - Pointers: `in` / `out` / `trace` are DEVICE pointers on the plan's device; every other
 *     pointer is HOST memory, read (or written) before the call returns.
 *   - Asynchrony: compute calls enqueue on `stream` (a hipStream_t passed as void*, NULL = the
 *     null stream) and return without synchronising.
 *   - Aliasing: in == out (in place) is allowed; any other overlap of the two extents is
 *     rejected with BSM_ERR_ALIAS.
 *   - Errors: every call returns a bsm_status; nothing is thrown, printed or aborted.  After a
 *     failure bsm_last_error() gives a thread-local description.  A failed call leaves its
 *     outputs untouched (no kernel is launched).  For tests of the failure paths, the
 *     environment variable BSM_TEST_ALLOC_FAIL makes every plan creation fail with
 *     BSM_ERR_OOM as if an allocation had failed: "host" after the table is built on the host,
 *     "device" at the device allocation of the work table (read at each plan creation).
 *   - Graph capture: an execution is one kernel launch that reads the plan's device table, so
 *     executions can be captured in a HIP graph; a plan must outlive every graph that captured
 *     one of its executions.
 *   - Element values: fp32, or bf16 (stored as raw 16-bit patterns); input and output share
 *     the type; arithmetic is fp32.  A row of all -inf (fully masked) yields zeros; a NaN or
 *     +inf entry makes its whole row NaN.
 */
#ifndef BSM_H
#define BSM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define BSM_ABI_VERSION 1
#define BSM_MAX_XCD 16

/* The enumerations' *_MAX_ENUM entries are not values: they make each enum a 32-bit type whose
 * range covers every int, so a caller passing any value is well-defined (and rejected with
 * BSM_ERR_INVALID_ARG when it names nothing). */
typedef enum bsm_status {
    BSM_OK = 0,
    BSM_ERR_INVALID_ARG = 1, /* bad pointer, size, enum, geometry or overlapping slices */
    BSM_ERR_UNSUPPORTED = 2, /* valid request the library cannot serve (e.g. host-only plan) */
    BSM_ERR_ALIAS = 3,       /* in and out overlap without being equal */
    BSM_ERR_OOM = 4,         /* host or device allocation failed */
    BSM_ERR_HIP = 5,         /* a HIP runtime call failed; bsm_last_error() has its string */
    BSM_STATUS_MAX_ENUM = 0x7FFFFFFF
} bsm_status;

typedef enum bsm_dtype { BSM_F32 = 0, BSM_BF16 = 1, BSM_DTYPE_MAX_ENUM = 0x7FFFFFFF } bsm_dtype;

/* Which worker processes which rows.
 *   RR        Section 3's prior solution: whole slice s goes to workgroup (s mod n_wg), whose
 *             waves share its rows.  Workers are workgroups.
 *   BALANCED  Section 4.2's load balancing at core granularity, with every wave a worker: the
 *             rows of all slices, in slice order, are cut into rounds of equal cost and every
 *             round into one piece per worker (pieces matched to the least-loaded workers), so
 *             each worker's total is within about one piece-granule of the MINIMAX optimum for
 *             this cost model and all workers sweep the tensor together.
 *   XCD       Sections 4.1 + 4.2: each slice gets a home XCD (the virtual bank holding the
 *             largest share of its elements, ties to the lowest index, or the caller's
 *             home_xcd[]); the load balancer moves the fewest rows it must from XCDs above
 *             their share to XCDs below it; each XCD's rows are then cut into rounds over the
 *             waves of that XCD's workgroups (workgroup w is planned for XCD w mod n_xcd:
 *             the dispatch order of MI355X, which now and then starts a launch on another
 *             XCD and so rotates the whole grid; results never depend on it). */
typedef enum bsm_schedule {
    BSM_SCHED_RR = 0,
    BSM_SCHED_BALANCED = 1,
    BSM_SCHED_XCD = 2,
    BSM_SCHED_MAX_ENUM = 0x7FFFFFFF
} bsm_schedule;

/* Launch geometry and cost model used by the planner.  Zero-filled fields take defaults. */
typedef struct bsm_topology {
    int32_t n_cu;        /* compute units (MI355X: 256) */
    int32_t n_xcd;       /* XCDs (MI355X: 8); workgroup w is taken to run on XCD w mod n_xcd */
    int32_t wg_per_cu;   /* persistent workgroups per CU; the grid has n_cu * wg_per_cu */
    int32_t wg_threads;  /* threads per workgroup, a multiple of 64 in [64, 1024]; plans with
                            rows longer than 2048 fp32 / 4096 bf16 elements run 256 (512 when
                            a row spans more than 16384 elements) whatever is asked: the
                            workgroup's waves share each such row; bf16 plans whose longest
                            row has 2049-4096 elements run at most 256 (their kernel needs
                            more registers than 1024-thread workgroups leave) */
    int32_t piece_bytes; /* BALANCED / XCD: traffic of one worker's piece of a round */
    float item_cost;     /* planner cost of one work item, in byte equivalents (<= 0: default) */
    float row_cost;      /* planner cost of one row on top of its bytes (<= 0: default) */
    int32_t flags;       /* BSM_FLAG_* bits; 0 = defaults */
} bsm_topology;

/* Cache policy.  By default rows are loaded and stored with nontemporal hints (streaming: best
 * for data that is not in any cache).  BSM_FLAG_TEMPORAL uses ordinary accesses instead, so
 * input that a producer kernel just wrote is served from the memory-side Infinity Cache
 * (256 MB on MI355X) and the output stays there for the consumer; use it when the batch fits.
 * Matrix-product plans take the same flag (C's stores and A's loads).  The output bits are the
 * same under both policies. */
#define BSM_FLAG_TEMPORAL 1

/* Virtual banks of the XCD schedule (Section 4.1's memory banks; MI355X in NPS1 interleaves HBM
 * over all stacks, so a bank is a planning construct).  By default the span of the non-empty
 * slices is cut into chunks dealt to the n_xcd banks in turn: a chunk is the mean slice extent
 * times the smallest factor that makes it at least 1 MiB (about one round of an XCD's workers),
 * so uniform slices of 1 MiB or more are homed on XCD s mod n_xcd.  Each XCD then streams a
 * contiguous chunk while the others stream the neighbouring ones.  When the
 * span holds no more than n_xcd chunks, or with BSM_FLAG_CONTIGUOUS_BANKS, the banks are n_xcd
 * equal contiguous ranges (the layout of Section 4.1's batch-to-bank table).  Homes change only
 * who computes a row: the output bits are the same. */
#define BSM_FLAG_CONTIGUOUS_BANKS 2

/* One entry of the work table (the paper's Patch<->Cluster mapping table, Section 5): `reps`
 * ranges of `nrows` rows each; range k starts at element elem_offset + k*rep_stride*cols.
 * Every row lies inside a slice of row length `cols` (a range may run on into the next slice
 * when the two are adjacent in memory and share the row length). */
typedef struct bsm_item {
    int64_t elem_offset; /* element offset of the first row of the first range */
    int32_t cols;        /* row length C, which is also the row stride */
    int32_t nrows;       /* rows per range */
    int32_t reps;        /* ranges (>= 1) */
    int32_t rep_stride;  /* rows from the start of one range to the start of the next */
    int32_t slice;       /* slice holding the item's first row */
    int32_t row_begin;   /* index of that row within its slice */
} bsm_item;

typedef struct bsm_plan_stats {
    int64_t batch;             /* slices */
    int64_t n_items;           /* entries of the work table */
    int64_t total_rows;        /* rows over all slices */
    int64_t algorithmic_bytes; /* every element read once plus written once */
    int64_t extent_elems;      /* elements from 0 to the end of the furthest slice */
    int64_t moved_bytes;       /* XCD: algorithmic bytes of rows run off their home XCD */
    int64_t trace_bytes;       /* size a trace buffer passed to bsm_plan_execute must have */
    int64_t n_rounds;          /* BALANCED / XCD: rounds the largest team's stream was cut into */
    int32_t n_workers;         /* entries of the work table's row pointer minus one */
    int32_t per_wave;          /* 1: workers are waves (w * waves_per_wg + wave); 0: workgroups
                                  (RR, and every plan with rows beyond the register tile) */
    int32_t n_wg;              /* persistent workgroups in the grid */
    int32_t n_xcd;
    int32_t wg_threads;
    int32_t schedule;          /* bsm_schedule */
    int32_t dtype;             /* bsm_dtype */
    int32_t n_overlap;         /* XCD: slices straddling two or more virtual banks */
    int32_t max_cols;          /* longest row */
    int32_t kernel_class;      /* which kernel instance the plan launches (internal) */
    int32_t lds_bytes_per_wave; /* LDS each wave may stage a row in (rows beyond the register
                                   tile whose start or length is not 16-byte aligned, and
                                   backward rows of 257..512 16-byte vectors; 0: none) */
    int32_t flags;             /* the BSM_FLAG_* bits the plan runs with */
    double max_worker_cost;    /* planner cost of the most loaded worker */
    double mean_worker_cost;   /* total planner cost / n_workers */
    double max_row_cost;       /* planner cost of the most expensive single row */
    double moved_cost;         /* XCD: planner cost of the rows run off their home XCD */
    double min_moved_cost;     /* XCD: sum over XCDs of (home load - fair share)+, the least
                                  any rebalancing must move */
    double build_us;           /* host time spent building the table */
    int64_t xcd_bytes[BSM_MAX_XCD];  /* algorithmic bytes run by each XCD's workgroups */
    int64_t bank_touch[BSM_MAX_XCD]; /* XCD: N_x, slices with elements in bank x */
    int64_t bank_home[BSM_MAX_XCD];  /* XCD: L_x, slices homed on bank x */
} bsm_plan_stats;

/* One record per wave when a trace buffer is passed to bsm_plan_execute (32 bytes). */
typedef struct bsm_trace_rec {
    uint32_t wg;      /* workgroup index in the grid */
    uint32_t xcc_id;  /* XCD the wave ran on, from the hardware XCC_ID register */
    uint32_t hw_id;   /* raw hardware HW_ID register (wave, SIMD, CU, shader engine) */
    uint32_t rows;    /* rows this wave processed (the one-pass score softmax of
                       * BSM_GEMM_NT_SOFTMAX: two waves share each row, the first counts it) */
    uint64_t t_start; /* constant-rate (100 MHz) real-time counter when the wave started */
    uint64_t t_end;   /* ... when it finished its last row */
} bsm_trace_rec;

typedef struct bsm_device_props {
    int32_t n_cu;
    int32_t n_xcd;
    int32_t wave_size;
    int32_t max_threads_per_cu;
    int64_t lds_bytes_per_cu;
    int64_t lds_bytes_per_wg;  /* largest LDS allocation of one workgroup */
    int64_t l2_bytes;          /* as reported by the runtime */
    int64_t hbm_bytes;
    int64_t wall_clock_hz;     /* rate of the counter in bsm_trace_rec */
    double peak_hbm_gbs;       /* from memory clock and bus width, as reported */
    int32_t clock_khz;
    char arch[64];             /* e.g. "gfx950:sramecc+:xnack-" */
} bsm_device_props;

typedef struct bsm_plan_s* bsm_plan;

/* One-shot batched row softmax.
 *   in, out        device buffers of `dtype` elements
 *   slice_offsets  NULL for uniform slices: then rows[0] = R and cols[0] = C for every slice
 *                  and slice s starts at element s*R*C.  Otherwise [batch] element offsets:
 *                  slice s occupies elements [slice_offsets[s], slice_offsets[s] + R_s*C_s).
 *                  Slices may sit in any order with gaps between them, but must not overlap;
 *                  gaps are never written.  A row that starts or ends inside a 16-byte
 *                  vector (buffers 16-byte aligned) is read as the aligned vectors that
 *                  cover it: up to 15 bytes before and after it are read and ignored (a
 *                  16-byte vector never crosses a page, so this cannot fault).
 *   rows, cols     [batch] (or [1] when uniform), each >= 0; an empty slice is skipped
 *   schedule       see bsm_schedule
 *   stream         hipStream_t as void*
 * Arguments are checked before any HIP call.  Plans are built on first use of a geometry and
 * cached per device (the 32 most recently used, plus any pinned by a graph capture); a later
 * call with the same arrays hashes and compares them and only launches the kernel.  No call
 * waits for the device: on a miss the plan is built on the host and its table uploaded with
 * hipMemcpyAsync on `stream` from pinned staging into a device buffer, both recycled by the
 * cache (evictions free nothing; a recycled buffer is ordered after its last readers by stream
 * waits on events, not by host waits).  Streams passed here must not be destroyed while work
 * they hold is still running.  Under stream capture a cached geometry is launched into the
 * graph and its plan is pinned until bsm_cache_clear; a geometry not in the cache returns
 * BSM_ERR_UNSUPPORTED (building a plan allocates and copies): run it once first.
 * batch == 0, or only empty slices, returns BSM_OK without touching the GPU. */
bsm_status bsm_softmax(const void* in, void* out, const int64_t* slice_offsets,
                       const int32_t* rows, const int32_t* cols, int64_t batch,
                       bsm_dtype dtype, bsm_schedule schedule, void* stream);

/* Size of the static device buffer of bsm_softmax_noalloc (per device). */
#define BSM_NOALLOC_SCRATCH_BYTES (8 * 1024 * 1024)

/* bsm_softmax for callers that cannot allocate device memory (hipMalloc is not allowed where
 * they run: tight serving loops, harnesses that forbid it).  Same arguments, checks and result
 * as bsm_softmax, but nothing is allocated on the device or pinned on the host and no plan is
 * cached: every call builds its plan on the host and copies its work table into a static
 * device buffer of BSM_NOALLOC_SCRATCH_BYTES bytes that the library holds on each device until
 * the process ends.  A plan whose table is larger (the call's message gives its size) returns
 * BSM_ERR_INVALID_ARG; BALANCED tables of the 384-slice workloads take 64 KiB (512 x 512
 * slices) to 3.4 MiB (ragged 64..1024-wide slices).  The copy is stream-ordered on `stream`
 * and the call returns once it has reached the device (it waits for the work queued before it
 * on `stream`); the kernel then runs asynchronously.  Every call on a device shares its
 * buffer: calls on one stream run in order, but calls that overlap on one device through
 * different streams or threads race (a later call may overwrite the table an earlier launch
 * is still reading).  Under stream capture it returns BSM_ERR_UNSUPPORTED. */
bsm_status bsm_softmax_noalloc(const void* in, void* out, const int64_t* slice_offsets,
                               const int32_t* rows, const int32_t* cols, int64_t batch,
                               bsm_dtype dtype, bsm_schedule schedule, void* stream);

/* Build a reusable plan: the work table of the HW batch scheduler of Section 5, built once
 * up front and reused for every execution.  The table is uploaded to the device before this
 * returns (synchronously).
 *   home_xcd   optional [batch] home XCD per slice in [0, n_xcd) for the XCD schedule (the
 *              bank each slice was created on); NULL = virtual banks over the span of the
 *              slices, interleaved chunks or contiguous ranges (BSM_FLAG_CONTIGUOUS_BANKS).
 *              Ignored by RR and BALANCED.
 *   topology   NULL = the device's defaults (bsm_default_topology).
 *   device     HIP device ordinal; -1 builds a host-only plan (topology required) that can
 *              be described and exported but not executed; it touches no GPU. */
bsm_status bsm_plan_create(bsm_plan* out_plan, const int64_t* slice_offsets,
                           const int32_t* rows, const int32_t* cols, int64_t batch,
                           bsm_dtype dtype, bsm_schedule schedule, const int8_t* home_xcd,
                           const bsm_topology* topology, int device);

/* bsm_plan_create with weighted load balancing (Section 4.2): under the XCD schedule, XCD x's
 * share of the total cost is proportional to (its workgroups) * xcd_weight[x] instead of to its
 * workgroups alone; the paper derives the weights from latencies, in inverse proportion, and
 * a caller can pass e.g. each XCD's measured throughput.  xcd_weight: NULL (equal weights, the
 * same table as bsm_plan_create) or [topology n_xcd] finite values >= 0, not all 0 (any
 * scale; an XCD of weight 0 receives no rows).  RR and BALANCED ignore the weights.  Other
 * arguments as bsm_plan_create; BSM_ERR_INVALID_ARG for bad weights. */
bsm_status bsm_plan_create_weighted(bsm_plan* out_plan, const int64_t* slice_offsets,
                                    const int32_t* rows, const int32_t* cols, int64_t batch,
                                    bsm_dtype dtype, bsm_schedule schedule,
                                    const int8_t* home_xcd, const float* xcd_weight,
                                    const bsm_topology* topology, int device);

/* Run a plan: out = row softmax of in, on `stream`.  `trace` is NULL or a device buffer of
 * stats.trace_bytes bytes that receives one bsm_trace_rec per wave. */
bsm_status bsm_plan_execute(bsm_plan plan, const void* in, void* out, void* stream, void* trace);

/* Softmax backward under a plan (the gradient pass that Section 1 says these batch
 * algorithms also run): for every row, with y the forward output and dy the gradient with
 * respect to y,
 *     d = sum_j dy_j * y_j,   dx_j = y_j * (dy_j - d)
 * (the softmax Jacobian diag(y) - y y^T applied to dy).  y, dy and dx are device buffers of the
 * plan's dtype and geometry; the arithmetic is fp32 (bf16 in and out rounds to nearest even).
 * dx may be y or dy exactly (in place); any other overlap of dx with an input is
 * BSM_ERR_ALIAS; y and dy may overlap freely.  Same table, stream and trace semantics as
 * bsm_plan_execute. */
bsm_status bsm_plan_execute_backward(bsm_plan plan, const void* y, const void* dy, void* dx,
                                     void* stream, void* trace);

/* One-shot softmax backward: the arguments of bsm_softmax, with y and dy in place of in and dx
 * in place of out; plans come from the same per-device cache. */
bsm_status bsm_softmax_backward(const void* y, const void* dy, void* dx,
                                const int64_t* slice_offsets, const int32_t* rows,
                                const int32_t* cols, int64_t batch, bsm_dtype dtype,
                                bsm_schedule schedule, void* stream);

/* ------------------------------------------------------------------ batched matrix products
 * The two batch matrix multiplications of Section 6 that surround the softmax in BERT
 * attention -- scores (512 x 64) x (64 x 512) and context (512 x 512) x (512 x 64), batch 384 --
 * scheduled by the same tables: the outputs C_b are the slices (m rows of n), cut by RR,
 * BALANCED or XCD as for the softmax, with one worker per workgroup (256 threads) and pieces
 * of whole 128-row blocks (the rows a workgroup takes per round, 32 per wave).
 *   BSM_GEMM_NT:  C_b = alpha * A_b * B_b^T    A_b m x k,  B_b n x k  (scores Q K^T)
 *   BSM_GEMM_NN:  C_b = alpha * A_b * B_b      A_b m x k,  B_b k x n  (context P V)
 * All operands row-major, batch after batch (A_b at b*m*k, B_b at b*n*k, C_b at b*m*n
 * elements).  A and B are bf16; C is fp32 or bf16 (round to nearest even); accumulation in
 * fp32 on the matrix cores. */
typedef enum {
    BSM_GEMM_NT = 0,
    BSM_GEMM_NN = 1,
    /* C_b = row softmax of alpha * A_b * B_b^T (A_b m x k, B_b n x k): Section 6's score
     * product followed by Section 2's softmax of every score row (each row of C_b sums to 1
     * over its n columns), in one kernel: the scores are never stored.  k == 0 gives rows
     * of 1/n.  For 0 < k <= 128 and 64 < n <= 512 (16-byte rows and operands, alpha != 0) each
     * product is formed once and held in registers until its row's sum is known; such plans
     * default to 2 workgroups per CU and take rounds of 64 rows (a topology asking for 3 or
     * more workgroups per CU keeps the two-pass form, whose rounds are 128 rows).  Otherwise
     * each round forms its products twice (row maximum and sum, then the probabilities). */
    BSM_GEMM_NT_SOFTMAX = 2,
    BSM_GEMM_LAYOUT_MAX_ENUM = 0x7FFFFFFF
} bsm_gemm_layout;

/* Build a matrix-product plan (out_dtype is C's type; home_xcd, topology and device as for
 * bsm_plan_create; topology->wg_threads must be 0 or 256, wg_per_cu defaults to 3, or to
 * 2 for the one-pass form of BSM_GEMM_NT_SOFTMAX).  A plan
 * made here runs only with bsm_gemm_execute.  Its stats report per_wave 0 (worker =
 * workgroup). */
bsm_status bsm_gemm_plan_create(bsm_plan* out_plan, int64_t batch, int32_t m, int32_t n,
                                int32_t k, bsm_gemm_layout layout, bsm_dtype out_dtype,
                                bsm_schedule schedule, const int8_t* home_xcd,
                                const bsm_topology* topology, int device);

/* C = alpha * product of A and B under the plan, on `stream` (asynchronous).  A, B, C are
 * device buffers; C must not overlap A or B (BSM_ERR_ALIAS).  k == 0 stores zeros.  `trace`
 * as for bsm_plan_execute (records count output rows). */
bsm_status bsm_gemm_execute(bsm_plan plan, const void* a, const void* b, void* c, float alpha,
                            void* stream, void* trace);

/* One-shot: plan from the per-device cache, then bsm_gemm_execute.  batch, m or n == 0 is a
 * no-op that touches no GPU. */
bsm_status bsm_gemm(const void* a, const void* b, void* c, int64_t batch, int32_t m, int32_t n,
                    int32_t k, bsm_gemm_layout layout, bsm_dtype out_dtype, float alpha,
                    bsm_schedule schedule, void* stream);

bsm_status bsm_plan_describe(bsm_plan plan, bsm_plan_stats* stats);

/* Copy the host work table out: worker_ptr [n_workers + 1] (CSR row pointer: worker v owns
 * items [worker_ptr[v], worker_ptr[v+1])), items [n_items], and, when non-NULL, home [batch]
 * (home XCD per slice after overlap resolution, -1 where the schedule has none) and overlap
 * [batch] (1 if the slice spans two or more virtual banks). */
bsm_status bsm_plan_export(bsm_plan plan, int32_t* worker_ptr, bsm_item* items, int8_t* home,
                           uint8_t* overlap);

/* Free a plan.  A plan that has been executed waits for its device to finish all queued work
 * first (executions record nothing per launch, so the wait is device-wide).  A plan may be
 * executed from several threads and streams, but must not be destroyed while another thread
 * executes it. */
bsm_status bsm_plan_destroy(bsm_plan plan);

bsm_status bsm_device_info(int device, bsm_device_props* info);

/* The topology bsm_plan_create uses for `device` when none is given. */
bsm_status bsm_default_topology(int device, bsm_topology* topology);

/* Plain device-to-device copy kernel of `bytes` bytes (128-bit accesses where aligned), the
 * streaming reference the softmax bandwidth is compared with.  src and dst must not overlap. */
bsm_status bsm_copy(const void* src, void* dst, int64_t bytes, void* stream);

/* Drop every cached one-shot plan and free the cache's device and pinned buffers: waits for
 * one-shot calls in other threads to finish launching, then for the device.  Graphs that
 * captured a one-shot call must not be replayed afterwards. */
bsm_status bsm_cache_clear(void);

const char* bsm_status_string(bsm_status status);
const char* bsm_last_error(void);
int32_t bsm_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* BSM_H */
