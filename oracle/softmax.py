"""ctypes wrapper of the fp64 C oracle (bsm_oracle.c).

TEST INFRASTRUCTURE ONLY: used by tests/, the smoke check and the bench's CPU-baseline leg.
It never imports the HIP library or its Python binding.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "bsm_oracle.c")
_LIB = os.path.join(_HERE, "libbsm_oracle.so")

DTYPE_CODE = {"f32": 0, "bf16": 1, "f64": 2}
_NP_DTYPE = {"f32": np.float32, "bf16": np.uint16, "f64": np.float64}

_lib = None


def build() -> str:
    """Compile libbsm_oracle.so with gcc (always recompiles)."""
    tmp = _LIB + ".tmp"
    cmd = ["gcc", "-O2", "-std=c99", "-Wall", "-Wextra", "-fPIC", "-shared", "-pthread",
           _SRC, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        i64p = ctypes.POINTER(ctypes.c_int64)
        i32p = ctypes.POINTER(ctypes.c_int32)
        f64p = ctypes.POINTER(ctypes.c_double)
        lib.bsm_oracle_softmax.argtypes = [ctypes.c_void_p, ctypes.c_int, i64p, i32p, i32p,
                                           ctypes.c_int64, f64p, ctypes.c_int]
        lib.bsm_oracle_softmax.restype = ctypes.c_int
        lib.bsm_oracle_softmax_rows.argtypes = [ctypes.c_void_p, ctypes.c_int, i64p, i32p,
                                                ctypes.c_int64, f64p]
        lib.bsm_oracle_softmax_rows.restype = ctypes.c_int
        lib.bsm_oracle_softmax_backward.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
                                                    i64p, i32p, i32p, ctypes.c_int64, f64p,
                                                    ctypes.c_int]
        lib.bsm_oracle_softmax_backward.restype = ctypes.c_int
        lib.bsm_oracle_softmax_backward_rows.argtypes = [ctypes.c_void_p, ctypes.c_void_p,
                                                         ctypes.c_int, i64p, i32p, ctypes.c_int64,
                                                         f64p]
        lib.bsm_oracle_softmax_backward_rows.restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _check_input(x: np.ndarray, dtype: str) -> np.ndarray:
    want = _NP_DTYPE[dtype]
    if x.dtype != want:
        raise TypeError(f"oracle input for {dtype} must be {np.dtype(want)}, got {x.dtype}")
    return np.ascontiguousarray(x.reshape(-1))


def softmax(x: np.ndarray, dtype: str, offsets, rows, cols, out: np.ndarray | None = None,
            nthreads: int = 1) -> np.ndarray:
    """fp64 row softmax of every row of every slice. Slice s has rows[s] x cols[s] elements
    starting at element offsets[s] of the flat input `x`. The fp64 output has the same element
    indexing as `x`; elements outside every slice keep the value they had in `out` (NaN when
    `out` is not given)."""
    x = _check_input(x, dtype)
    offsets = np.ascontiguousarray(offsets, dtype=np.int64)
    rows = np.ascontiguousarray(rows, dtype=np.int32)
    cols = np.ascontiguousarray(cols, dtype=np.int32)
    batch = int(rows.shape[0])
    if offsets.shape[0] < batch or cols.shape[0] != batch:
        raise ValueError("offsets/rows/cols lengths disagree")
    if batch:
        end = int(np.max(offsets[:batch] + rows.astype(np.int64) * cols.astype(np.int64)))
        if end > x.shape[0]:
            raise ValueError("a slice extends past the end of the input")
    if out is None:
        out = np.full(x.shape[0], np.nan, dtype=np.float64)
    if out.dtype != np.float64 or out.shape[0] < x.shape[0] or not out.flags.c_contiguous:
        raise ValueError("out must be a contiguous float64 array at least as long as x")
    rc = _load().bsm_oracle_softmax(x.ctypes.data, DTYPE_CODE[dtype], _ptr(offsets, ctypes.c_int64),
                                    _ptr(rows, ctypes.c_int32), _ptr(cols, ctypes.c_int32),
                                    batch, _ptr(out, ctypes.c_double), int(nthreads))
    if rc != 0:
        raise ValueError("oracle rejected its arguments")
    return out


def softmax_rows(x: np.ndarray, dtype: str, row_first, row_cols) -> np.ndarray:
    """fp64 softmax of selected rows: row i has row_cols[i] elements starting at element
    row_first[i] of `x`. Returns the rows concatenated in order."""
    x = _check_input(x, dtype)
    row_first = np.ascontiguousarray(row_first, dtype=np.int64)
    row_cols = np.ascontiguousarray(row_cols, dtype=np.int32)
    n = int(row_first.shape[0])
    if n and int(np.max(row_first + row_cols)) > x.shape[0]:
        raise ValueError("a row extends past the end of the input")
    out = np.empty(int(np.sum(row_cols, dtype=np.int64)), dtype=np.float64)
    rc = _load().bsm_oracle_softmax_rows(x.ctypes.data, DTYPE_CODE[dtype],
                                         _ptr(row_first, ctypes.c_int64),
                                         _ptr(row_cols, ctypes.c_int32), n,
                                         _ptr(out, ctypes.c_double))
    if rc != 0:
        raise ValueError("oracle rejected its arguments")
    return out


def softmax_backward(y: np.ndarray, dy: np.ndarray, dtype: str, offsets, rows, cols,
                     out: np.ndarray | None = None, nthreads: int = 1) -> np.ndarray:
    """fp64 softmax backward of every row of every slice: dx = y * (dy - sum(dy * y)) per row,
    from the forward output `y` and the gradient `dy` (same dtype and element indexing). Same
    slice arguments and output convention as `softmax`."""
    y = _check_input(y, dtype)
    dy = _check_input(dy, dtype)
    if y.shape != dy.shape:
        raise ValueError("y and dy must have the same length")
    offsets = np.ascontiguousarray(offsets, dtype=np.int64)
    rows = np.ascontiguousarray(rows, dtype=np.int32)
    cols = np.ascontiguousarray(cols, dtype=np.int32)
    batch = int(rows.shape[0])
    if offsets.shape[0] < batch or cols.shape[0] != batch:
        raise ValueError("offsets/rows/cols lengths disagree")
    if batch:
        end = int(np.max(offsets[:batch] + rows.astype(np.int64) * cols.astype(np.int64)))
        if end > y.shape[0]:
            raise ValueError("a slice extends past the end of the input")
    if out is None:
        out = np.full(y.shape[0], np.nan, dtype=np.float64)
    if out.dtype != np.float64 or out.shape[0] < y.shape[0] or not out.flags.c_contiguous:
        raise ValueError("out must be a contiguous float64 array at least as long as y")
    rc = _load().bsm_oracle_softmax_backward(
        y.ctypes.data, dy.ctypes.data, DTYPE_CODE[dtype], _ptr(offsets, ctypes.c_int64),
        _ptr(rows, ctypes.c_int32), _ptr(cols, ctypes.c_int32), batch,
        _ptr(out, ctypes.c_double), int(nthreads))
    if rc != 0:
        raise ValueError("oracle rejected its arguments")
    return out


def softmax_backward_rows(y: np.ndarray, dy: np.ndarray, dtype: str, row_first,
                          row_cols) -> np.ndarray:
    """fp64 softmax backward of selected rows (as `softmax_rows`)."""
    y = _check_input(y, dtype)
    dy = _check_input(dy, dtype)
    if y.shape != dy.shape:
        raise ValueError("y and dy must have the same length")
    row_first = np.ascontiguousarray(row_first, dtype=np.int64)
    row_cols = np.ascontiguousarray(row_cols, dtype=np.int32)
    n = int(row_first.shape[0])
    if n and int(np.max(row_first + row_cols)) > y.shape[0]:
        raise ValueError("a row extends past the end of the input")
    out = np.empty(int(np.sum(row_cols, dtype=np.int64)), dtype=np.float64)
    rc = _load().bsm_oracle_softmax_backward_rows(
        y.ctypes.data, dy.ctypes.data, DTYPE_CODE[dtype], _ptr(row_first, ctypes.c_int64),
        _ptr(row_cols, ctypes.c_int32), n, _ptr(out, ctypes.c_double))
    if rc != 0:
        raise ValueError("oracle rejected its arguments")
    return out
