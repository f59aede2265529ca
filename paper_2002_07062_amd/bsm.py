"""ctypes binding of libbsm.so: the same entry points as include/bsm.h.

Argument marshalling only: tensors become device pointers, metadata becomes host arrays, the
stream is torch's current stream on the tensor's device. Every computation runs in the HIP
kernels of libbsm.so; there is no fallback, and a missing library raises at load time.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np

# torch first: libbsm.so then binds to the HIP runtime torch has already loaded (both carry
# the same SONAME), so tensors, streams and kernels share one runtime.
import torch

# the in-tree build; BSM_LIB names another build of the same library (e.g. one with host-side
# sanitizers for the CPU tests)
LIB_PATH = os.environ.get("BSM_LIB") or os.path.join(os.path.dirname(os.path.abspath(__file__)), "libbsm.so")

BSM_OK, BSM_ERR_INVALID_ARG, BSM_ERR_UNSUPPORTED, BSM_ERR_ALIAS, BSM_ERR_OOM, BSM_ERR_HIP = range(6)
BSM_F32, BSM_BF16 = 0, 1
BSM_SCHED_RR, BSM_SCHED_BALANCED, BSM_SCHED_XCD = 0, 1, 2
BSM_MAX_XCD = 16
BSM_NOALLOC_SCRATCH_BYTES = 8 * 1024 * 1024  # static buffer of bsm_softmax_noalloc
BSM_FLAG_TEMPORAL = 1
BSM_FLAG_CONTIGUOUS_BANKS = 2

SCHEDULES = {"rr": BSM_SCHED_RR, "balanced": BSM_SCHED_BALANCED, "xcd": BSM_SCHED_XCD}
BSM_GEMM_NT, BSM_GEMM_NN, BSM_GEMM_NT_SOFTMAX = 0, 1, 2
# "nt_softmax": C = row softmax of alpha A B^T (the score product and the softmax in one kernel)
GEMM_LAYOUTS = {"nt": BSM_GEMM_NT, "nn": BSM_GEMM_NN, "nt_softmax": BSM_GEMM_NT_SOFTMAX}
DTYPES = {"f32": BSM_F32, "bf16": BSM_BF16}


class BsmError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{_STATUS_NAMES.get(status, status)}: {message}")
        self.status = status
        self.message = message


_STATUS_NAMES = {0: "BSM_OK", 1: "BSM_ERR_INVALID_ARG", 2: "BSM_ERR_UNSUPPORTED",
                 3: "BSM_ERR_ALIAS", 4: "BSM_ERR_OOM", 5: "BSM_ERR_HIP"}


class bsm_topology(ctypes.Structure):
    _fields_ = [("n_cu", ctypes.c_int32), ("n_xcd", ctypes.c_int32),
                ("wg_per_cu", ctypes.c_int32), ("wg_threads", ctypes.c_int32),
                ("piece_bytes", ctypes.c_int32), ("item_cost", ctypes.c_float),
                ("row_cost", ctypes.c_float), ("flags", ctypes.c_int32)]


class bsm_item(ctypes.Structure):
    _fields_ = [("elem_offset", ctypes.c_int64), ("cols", ctypes.c_int32),
                ("nrows", ctypes.c_int32), ("reps", ctypes.c_int32),
                ("rep_stride", ctypes.c_int32), ("slice", ctypes.c_int32),
                ("row_begin", ctypes.c_int32)]


ITEM_DTYPE = np.dtype([("elem_offset", "<i8"), ("cols", "<i4"), ("nrows", "<i4"),
                       ("reps", "<i4"), ("rep_stride", "<i4"), ("slice", "<i4"),
                       ("row_begin", "<i4")])
TRACE_DTYPE = np.dtype([("wg", "<u4"), ("xcc_id", "<u4"), ("hw_id", "<u4"), ("rows", "<u4"),
                        ("t_start", "<u8"), ("t_end", "<u8")])


class bsm_plan_stats(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int64), ("n_items", ctypes.c_int64),
                ("total_rows", ctypes.c_int64), ("algorithmic_bytes", ctypes.c_int64),
                ("extent_elems", ctypes.c_int64), ("moved_bytes", ctypes.c_int64),
                ("trace_bytes", ctypes.c_int64), ("n_rounds", ctypes.c_int64),
                ("n_workers", ctypes.c_int32), ("per_wave", ctypes.c_int32),
                ("n_wg", ctypes.c_int32), ("n_xcd", ctypes.c_int32),
                ("wg_threads", ctypes.c_int32), ("schedule", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("n_overlap", ctypes.c_int32),
                ("max_cols", ctypes.c_int32), ("kernel_class", ctypes.c_int32),
                ("lds_bytes_per_wave", ctypes.c_int32), ("flags", ctypes.c_int32),
                ("max_worker_cost", ctypes.c_double), ("mean_worker_cost", ctypes.c_double),
                ("max_row_cost", ctypes.c_double), ("moved_cost", ctypes.c_double),
                ("min_moved_cost", ctypes.c_double), ("build_us", ctypes.c_double),
                ("xcd_bytes", ctypes.c_int64 * BSM_MAX_XCD),
                ("bank_touch", ctypes.c_int64 * BSM_MAX_XCD),
                ("bank_home", ctypes.c_int64 * BSM_MAX_XCD)]


class bsm_device_props(ctypes.Structure):
    _fields_ = [("n_cu", ctypes.c_int32), ("n_xcd", ctypes.c_int32),
                ("wave_size", ctypes.c_int32), ("max_threads_per_cu", ctypes.c_int32),
                ("lds_bytes_per_cu", ctypes.c_int64), ("lds_bytes_per_wg", ctypes.c_int64),
                ("l2_bytes", ctypes.c_int64),
                ("hbm_bytes", ctypes.c_int64), ("wall_clock_hz", ctypes.c_int64),
                ("peak_hbm_gbs", ctypes.c_double), ("clock_khz", ctypes.c_int32),
                ("arch", ctypes.c_char * 64)]


_lib = None


def load() -> ctypes.CDLL:
    """Load libbsm.so (built by `python -m paper_2002_07062_amd.build`). Raises if missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2002_07062_amd.build` "
                           "(or __graft_entry__.build()) first")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    P = ctypes.POINTER
    sig = {
        "bsm_softmax": ([vp, vp, P(i64), P(i32), P(i32), i64, ctypes.c_int, ctypes.c_int, vp],
                        ctypes.c_int),
        "bsm_softmax_noalloc": ([vp, vp, P(i64), P(i32), P(i32), i64, ctypes.c_int, ctypes.c_int,
                                 vp], ctypes.c_int),
        "bsm_plan_create": ([P(vp), P(i64), P(i32), P(i32), i64, ctypes.c_int, ctypes.c_int,
                             P(ctypes.c_int8), P(bsm_topology), ctypes.c_int], ctypes.c_int),
        "bsm_plan_create_weighted": ([P(vp), P(i64), P(i32), P(i32), i64, ctypes.c_int,
                                      ctypes.c_int, P(ctypes.c_int8), P(ctypes.c_float),
                                      P(bsm_topology), ctypes.c_int], ctypes.c_int),
        "bsm_plan_execute": ([vp, vp, vp, vp, vp], ctypes.c_int),
        "bsm_gemm_plan_create": ([P(vp), i64, i32, i32, i32, ctypes.c_int, ctypes.c_int,
                                  ctypes.c_int, P(ctypes.c_int8), P(bsm_topology), ctypes.c_int],
                                 ctypes.c_int),
        "bsm_gemm_execute": ([vp, vp, vp, vp, ctypes.c_float, vp, vp], ctypes.c_int),
        "bsm_gemm": ([vp, vp, vp, i64, i32, i32, i32, ctypes.c_int, ctypes.c_int, ctypes.c_float,
                      ctypes.c_int, vp], ctypes.c_int),
        "bsm_plan_execute_backward": ([vp, vp, vp, vp, vp, vp], ctypes.c_int),
        "bsm_softmax_backward": ([vp, vp, vp, P(i64), P(i32), P(i32), i64, ctypes.c_int,
                                  ctypes.c_int, vp], ctypes.c_int),
        "bsm_plan_describe": ([vp, P(bsm_plan_stats)], ctypes.c_int),
        "bsm_plan_export": ([vp, P(i32), vp, P(ctypes.c_int8), P(ctypes.c_uint8)], ctypes.c_int),
        "bsm_plan_destroy": ([vp], ctypes.c_int),
        "bsm_device_info": ([ctypes.c_int, P(bsm_device_props)], ctypes.c_int),
        "bsm_default_topology": ([ctypes.c_int, P(bsm_topology)], ctypes.c_int),
        "bsm_copy": ([vp, vp, i64, vp], ctypes.c_int),
        "bsm_cache_clear": ([], ctypes.c_int),
        "bsm_status_string": ([ctypes.c_int], ctypes.c_char_p),
        "bsm_last_error": ([], ctypes.c_char_p),
        "bsm_abi_version": ([], i32),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def _check(status: int) -> None:
    if status != BSM_OK:
        raise BsmError(status, load().bsm_last_error().decode(errors="replace"))


def _arr(a, dtype):
    if a is None:
        return None, None
    arr = np.ascontiguousarray(np.asarray(a), dtype=dtype).reshape(-1)
    return arr, arr.ctypes.data_as(ctypes.POINTER(np.ctypeslib.as_ctypes_type(dtype)))


def _dtype_code(d) -> int:
    if isinstance(d, str):
        return DTYPES[d]
    if isinstance(d, (int, np.integer)):
        return int(d)  # raw bsm_dtype code: the library validates it
    if d == torch.float32:
        return BSM_F32
    if d == torch.bfloat16:
        return BSM_BF16
    raise TypeError(f"unsupported dtype {d}: float32 or bfloat16")


def _schedule_code(s) -> int:
    return SCHEDULES[s] if isinstance(s, str) else int(s)


def _ptr(t) -> int | None:
    if t is None:
        return None
    if isinstance(t, torch.Tensor):
        if not t.is_cuda:
            raise ValueError("expected a GPU tensor")
        if not t.is_contiguous():
            raise ValueError("expected a contiguous tensor")
        return t.data_ptr()
    return int(t)


def _stream_of(t, stream):
    if stream is not None:
        return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
    if isinstance(t, torch.Tensor) and t.is_cuda:
        return torch.cuda.current_stream(t.device).cuda_stream
    return None


def _geometry(rows, cols, slice_offsets, batch):
    """Uniform when slice_offsets is None (rows/cols scalars, batch required), else per-slice
    arrays whose length is the batch."""
    if slice_offsets is None:
        if batch is None:
            raise ValueError("uniform geometry needs batch")
        r, rp = _arr([int(np.asarray(rows).reshape(-1)[0])], np.int32)
        c, cp = _arr([int(np.asarray(cols).reshape(-1)[0])], np.int32)
        return None, None, r, rp, c, cp, int(batch)
    o, op = _arr(slice_offsets, np.int64)
    r, rp = _arr(rows, np.int32)
    c, cp = _arr(cols, np.int32)
    n = int(r.shape[0]) if batch is None else int(batch)
    if o.shape[0] < n or r.shape[0] < n or c.shape[0] < n:
        raise ValueError("slice_offsets/rows/cols shorter than batch")
    return o, op, r, rp, c, cp, n


def _extent(o, r, c, n) -> int:
    """Elements from 0 to the end of the furthest non-empty slice."""
    if n == 0:
        return 0
    if o is None:
        return int(r[0]) * int(c[0]) * n
    sizes = r[:n].astype(np.int64) * c[:n].astype(np.int64)
    live = sizes > 0
    return int(np.max(o[:n][live] + sizes[live])) if live.any() else 0


def _check_sizes(extent: int, *tensors) -> None:
    for t in tensors:
        if isinstance(t, torch.Tensor) and t.numel() < extent:
            raise ValueError(f"tensor of {t.numel()} elements is shorter than the slices' "
                             f"extent ({extent} elements)")


def bsm_softmax(x, out, rows, cols, slice_offsets=None, batch=None, schedule="balanced",
                stream=None):
    """out = row softmax of x over every slice (see bsm.h). x, out: contiguous GPU tensors of
    float32 or bfloat16 (out may be x). Returns out."""
    lib = load()
    if out.dtype != x.dtype:
        raise TypeError("x and out must share a dtype")
    keep = _geometry(rows, cols, slice_offsets, batch)
    o, op, r, rp, c, cp, n = keep
    _check_sizes(_extent(o, r, c, n), x, out)
    with torch.cuda.device(x.device):
        _check(lib.bsm_softmax(_ptr(x), _ptr(out), op, rp, cp, n, _dtype_code(x.dtype),
                               _schedule_code(schedule), _stream_of(x, stream)))
    return out


def bsm_softmax_noalloc(x, out, rows, cols, slice_offsets=None, batch=None, schedule="balanced",
                        stream=None):
    """bsm_softmax with the work table in the library's static device buffer (no device or
    pinned allocation; see bsm.h). Returns out."""
    lib = load()
    if out.dtype != x.dtype:
        raise TypeError("x and out must share a dtype")
    keep = _geometry(rows, cols, slice_offsets, batch)
    o, op, r, rp, c, cp, n = keep
    _check_sizes(_extent(o, r, c, n), x, out)
    with torch.cuda.device(x.device):
        _check(lib.bsm_softmax_noalloc(_ptr(x), _ptr(out), op, rp, cp, n, _dtype_code(x.dtype),
                                       _schedule_code(schedule), _stream_of(x, stream)))
    return out


def bsm_softmax_backward(y, dy, dx, rows, cols, slice_offsets=None, batch=None,
                         schedule="balanced", stream=None):
    """dx = softmax backward of (y, dy) over every slice: per row d = sum(dy * y),
    dx = y * (dy - d) (see bsm.h). y, dy, dx: contiguous GPU tensors of one dtype (dx may be y
    or dy). Returns dx."""
    lib = load()
    if not (y.dtype == dy.dtype == dx.dtype):
        raise TypeError("y, dy and dx must share a dtype")
    keep = _geometry(rows, cols, slice_offsets, batch)
    o, op, r, rp, c, cp, n = keep
    _check_sizes(_extent(o, r, c, n), y, dy, dx)
    with torch.cuda.device(y.device):
        _check(lib.bsm_softmax_backward(_ptr(y), _ptr(dy), _ptr(dx), op, rp, cp, n,
                                        _dtype_code(y.dtype), _schedule_code(schedule),
                                        _stream_of(y, stream)))
    return dx


class Plan:
    """A built work table (bsm_plan). Use bsm_plan_create to make one."""

    def __init__(self, handle: int, batch: int, device: int, extent: int, trace_bytes: int,
                 dtype: int = BSM_F32):
        self.handle = handle
        self.batch = batch
        self.device = device
        self.extent = extent
        self.trace_bytes = trace_bytes
        self.dtype = dtype

    def check_tensors(self, *tensors) -> None:
        """Every tensor covers the plan's extent and has the plan's element type."""
        _check_sizes(self.extent, *tensors)
        want = torch.float32 if self.dtype == BSM_F32 else torch.bfloat16
        for t in tensors:
            if isinstance(t, torch.Tensor) and t.dtype != want:
                raise TypeError(f"plan is for {want}, got a {t.dtype} tensor")

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.destroy()

    def destroy(self):
        if self.handle:
            h, self.handle = self.handle, None
            _check(load().bsm_plan_destroy(h))

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


def bsm_plan_create(rows, cols, slice_offsets=None, batch=None, dtype="f32", schedule="balanced",
                    home_xcd=None, topology=None, device=0, xcd_weight=None) -> Plan:
    """Build a plan. `topology`: None, a bsm_topology or a dict of its fields. device=-1 makes
    a host-only plan (needs a topology) that can be described and exported but not run.
    `xcd_weight`: None or one weight per XCD (bsm_plan_create_weighted)."""
    lib = load()
    _, op, _, rp, _, cp, n = keep = _geometry(rows, cols, slice_offsets, batch)
    h, hp = _arr(home_xcd, np.int8)
    wt, wp = _arr(xcd_weight, np.float32)
    topo = None
    if topology is not None:
        topo = topology if isinstance(topology, bsm_topology) else bsm_topology(**topology)
    if xcd_weight is not None:
        n_xcd = topo.n_xcd if topo is not None and topo.n_xcd > 0 else (
            bsm_default_topology(int(device))["n_xcd"] if int(device) >= 0 else 8)
        if wt.shape[0] != n_xcd:
            raise ValueError(f"xcd_weight needs {n_xcd} entries (one per XCD), got {wt.shape[0]}")
    handle = ctypes.c_void_p()
    tp = ctypes.byref(topo) if topo is not None else None
    if xcd_weight is None:
        _check(lib.bsm_plan_create(ctypes.byref(handle), op, rp, cp, n, _dtype_code(dtype),
                                   _schedule_code(schedule), hp, tp, int(device)))
    else:
        _check(lib.bsm_plan_create_weighted(ctypes.byref(handle), op, rp, cp, n,
                                            _dtype_code(dtype), _schedule_code(schedule), hp, wp,
                                            tp, int(device)))
    del keep, h, wt
    st = bsm_plan_stats()
    _check(lib.bsm_plan_describe(handle.value, ctypes.byref(st)))
    return Plan(handle.value, n, int(device), int(st.extent_elems), int(st.trace_bytes),
                int(st.dtype))


def bsm_plan_execute(plan: Plan, x, out, stream=None, trace=None):
    """out = row softmax of x under the plan. `trace`: None or a GPU tensor of at least
    stats['trace_bytes'] bytes (one TRACE_DTYPE record per wave)."""
    lib = load()
    plan.check_tensors(x, out)
    if trace is not None and trace.numel() * trace.element_size() < plan.trace_bytes:
        raise ValueError(f"trace buffer needs {plan.trace_bytes} bytes")
    with torch.cuda.device(plan.device):
        _check(lib.bsm_plan_execute(plan.handle, _ptr(x), _ptr(out), _stream_of(x, stream),
                                    _ptr(trace)))
    return out


def bsm_plan_execute_backward(plan: Plan, y, dy, dx, stream=None, trace=None):
    """dx = softmax backward of (y, dy) under the plan (same geometry and dtype as its
    forward). `trace` as for bsm_plan_execute."""
    lib = load()
    plan.check_tensors(y, dy, dx)
    if trace is not None and trace.numel() * trace.element_size() < plan.trace_bytes:
        raise ValueError(f"trace buffer needs {plan.trace_bytes} bytes")
    with torch.cuda.device(plan.device):
        _check(lib.bsm_plan_execute_backward(plan.handle, _ptr(y), _ptr(dy), _ptr(dx),
                                             _stream_of(y, stream), _ptr(trace)))
    return dx


def bsm_plan_describe(plan: Plan) -> dict:
    st = bsm_plan_stats()
    _check(load().bsm_plan_describe(plan.handle, ctypes.byref(st)))
    d = {}
    for name, _ in bsm_plan_stats._fields_:
        v = getattr(st, name)
        d[name] = list(v)[: st.n_xcd] if name in ("xcd_bytes", "bank_touch", "bank_home") else v
    return d


def bsm_plan_export(plan: Plan):
    """Returns (worker_ptr int32[n_workers+1], items ITEM_DTYPE[n_items], home int8[batch],
    overlap uint8[batch])."""
    d = bsm_plan_describe(plan)
    wg_ptr = np.zeros(d["n_workers"] + 1, np.int32)
    items = np.zeros(d["n_items"], ITEM_DTYPE)
    home = np.zeros(plan.batch, np.int8)
    overlap = np.zeros(plan.batch, np.uint8)
    _check(load().bsm_plan_export(plan.handle, wg_ptr.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                  items.ctypes.data if len(items) else None,
                                  home.ctypes.data_as(ctypes.POINTER(ctypes.c_int8)),
                                  overlap.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8))))
    return wg_ptr, items, home, overlap


def bsm_plan_destroy(plan: Plan) -> None:
    plan.destroy()


def bsm_device_info(device: int = 0) -> dict:
    p = bsm_device_props()
    _check(load().bsm_device_info(int(device), ctypes.byref(p)))
    d = {name: getattr(p, name) for name, _ in bsm_device_props._fields_}
    d["arch"] = p.arch.decode(errors="replace")
    return d


def bsm_default_topology(device: int = 0) -> dict:
    t = bsm_topology()
    _check(load().bsm_default_topology(int(device), ctypes.byref(t)))
    return {name: getattr(t, name) for name, _ in bsm_topology._fields_}


def bsm_copy(src, dst, nbytes=None, stream=None):
    """dst[:nbytes] = src[:nbytes] with the library's streaming copy kernel."""
    if nbytes is None:
        nbytes = min(src.numel() * src.element_size(), dst.numel() * dst.element_size())
    with torch.cuda.device(src.device):
        _check(load().bsm_copy(_ptr(src), _ptr(dst), int(nbytes), _stream_of(src, stream)))
    return dst


def bsm_cache_clear() -> None:
    _check(load().bsm_cache_clear())


def bsm_status_string(status: int) -> str:
    return load().bsm_status_string(int(status)).decode()


def bsm_last_error() -> str:
    return load().bsm_last_error().decode(errors="replace")


def bsm_abi_version() -> int:
    return int(load().bsm_abi_version())


# ------------------------------------------------------------------ batched matrix products
def _layout_code(layout) -> int:
    if isinstance(layout, int):
        return layout
    return GEMM_LAYOUTS[layout]


def _check_gemm_tensors(batch, m, n, k, a, b, c, c_dtype) -> None:
    for t, need, name in ((a, batch * m * k, "a"), (b, batch * n * k, "b"), (c, batch * m * n, "c")):
        if t.numel() < need:
            raise ValueError(f"{name} has {t.numel()} elements, needs {need}")
    if a.dtype != torch.bfloat16 or b.dtype != torch.bfloat16:
        raise TypeError("a and b must be bfloat16")
    if c.dtype != c_dtype:
        raise TypeError(f"c must be {c_dtype}")


def bsm_gemm_plan_create(batch, m, n, k, layout="nt", out_dtype="f32", schedule="balanced",
                         home_xcd=None, topology=None, device=0) -> Plan:
    """Plan of the batched product C_b = alpha A_b B_b^T ("nt"), alpha A_b B_b ("nn"), or the
    row softmax of alpha A_b B_b^T ("nt_softmax")."""
    lib = load()
    h, hp = _arr(home_xcd, np.int8)
    topo = None
    if topology is not None:
        topo = topology if isinstance(topology, bsm_topology) else bsm_topology(**topology)
    handle = ctypes.c_void_p()
    _check(lib.bsm_gemm_plan_create(ctypes.byref(handle), int(batch), int(m), int(n), int(k),
                                    _layout_code(layout), _dtype_code(out_dtype),
                                    _schedule_code(schedule), hp,
                                    ctypes.byref(topo) if topo is not None else None, int(device)))
    del h
    st = bsm_plan_stats()
    _check(lib.bsm_plan_describe(handle.value, ctypes.byref(st)))
    plan = Plan(handle.value, int(batch), int(device), 0, int(st.trace_bytes), int(st.dtype))
    plan.gemm = (int(batch), int(m), int(n), int(k))
    return plan


def bsm_gemm_execute(plan: Plan, a, b, c, alpha=1.0, stream=None, trace=None):
    """c = product of a and b under the plan (see bsm.h). Returns c."""
    lib = load()
    batch, m, n, k = plan.gemm
    _check_gemm_tensors(batch, m, n, k, a, b, c,
                        torch.float32 if plan.dtype == BSM_F32 else torch.bfloat16)
    if trace is not None and trace.numel() * trace.element_size() < plan.trace_bytes:
        raise ValueError(f"trace buffer needs {plan.trace_bytes} bytes")
    with torch.cuda.device(plan.device):
        _check(lib.bsm_gemm_execute(plan.handle, _ptr(a), _ptr(b), _ptr(c), float(alpha),
                                    _stream_of(c, stream), _ptr(trace)))
    return c


def bsm_gemm(a, b, c, batch, m, n, k, layout="nt", alpha=1.0, schedule="balanced", stream=None):
    """One-shot batched product (plans cached per device). c's dtype picks fp32 or bf16 output."""
    lib = load()
    _check_gemm_tensors(batch, m, n, k, a, b, c, c.dtype)
    with torch.cuda.device(c.device):
        _check(lib.bsm_gemm(_ptr(a), _ptr(b), _ptr(c), int(batch), int(m), int(n), int(k),
                            _layout_code(layout), _dtype_code(c.dtype), float(alpha),
                            _schedule_code(schedule), _stream_of(c, stream)))
    return c
