"""fp64 oracle of the batched matrix products around the softmax (Section 6's two batch matrix
multiplications of BERT: (512 x 64) x (64 x 512) and (512 x 512) x (512 x 64), batch 384).

TEST INFRASTRUCTURE ONLY: used by tests/, the smoke check and the bench's CPU-baseline leg. It
shares no code with the HIP library.

What it computes, for every batch index b (each operand stored row-major, batch after batch):

    layout "nt":  C_b = alpha * A_b @ B_b^T     A_b: m x k,  B_b: n x k,  C_b: m x n
    layout "nn":  C_b = alpha * A_b @ B_b       A_b: m x k,  B_b: k x n,  C_b: m x n

    layout "nt_softmax": C_b = row softmax of (alpha * A_b @ B_b^T)

"nt" is the score product Q K^T of attention (keys stored one per row); "nn" is the context
product P V; "nt_softmax" is the score product followed by Section 2's softmax of every score
row (scores_softmax below: this module's product, then the softmax oracle of oracle/softmax.py
over the batch * m rows of n values). Operands are bf16 bit patterns (or fp32 / fp64 values), converted to fp64
exactly; the product of each batch is numpy's fp64 matrix product (a library primitive),
then scaled by alpha in fp64.
"""

from __future__ import annotations

import numpy as np

LAYOUTS = ("nt", "nn")


def _to_f64(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        if x.dtype != np.uint16:
            raise TypeError("bf16 operands are uint16 bit patterns")
        return (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    if dtype == "f32":
        if x.dtype != np.float32:
            raise TypeError("f32 operands must be float32")
        return x.astype(np.float64)
    if dtype == "f64":
        return np.asarray(x, np.float64)
    raise ValueError(f"unknown dtype {dtype}")


def batched_gemm(a: np.ndarray, b: np.ndarray, batch: int, m: int, n: int, k: int,
                 layout: str = "nt", alpha: float = 1.0, dtype: str = "bf16") -> np.ndarray:
    """fp64 C (batch * m * n, row-major per batch) of the batched product described above."""
    if layout not in LAYOUTS:
        raise ValueError(f"layout must be one of {LAYOUTS}")
    if min(batch, m, n, k) < 0:
        raise ValueError("negative size")
    A = _to_f64(np.ascontiguousarray(a).reshape(-1), dtype)
    B = _to_f64(np.ascontiguousarray(b).reshape(-1), dtype)
    if A.shape[0] < batch * m * k or B.shape[0] < batch * n * k:
        raise ValueError("operand shorter than batch * rows * cols")
    A = A[: batch * m * k].reshape(batch, m, k)
    if layout == "nt":
        Bt = B[: batch * n * k].reshape(batch, n, k).transpose(0, 2, 1)
    else:
        Bt = B[: batch * n * k].reshape(batch, k, n)
    C = np.empty((batch, m, n), np.float64)
    for i in range(batch):
        C[i] = A[i] @ Bt[i]
    return (C * float(alpha)).reshape(-1)


def abs_product_sums(a: np.ndarray, b: np.ndarray, batch: int, m: int, n: int, k: int,
                     layout: str = "nt", dtype: str = "bf16") -> np.ndarray:
    """sum_k |a_ik| |b_kj| for every output element (the scale of its rounding error)."""
    A = np.abs(_to_f64(np.ascontiguousarray(a).reshape(-1), dtype))
    B = np.abs(_to_f64(np.ascontiguousarray(b).reshape(-1), dtype))
    return batched_gemm(A, B, batch, m, n, k, layout, 1.0, "f64")


def scores_softmax(a: np.ndarray, b: np.ndarray, batch: int, m: int, n: int, k: int,
                   alpha: float = 1.0, dtype: str = "bf16") -> np.ndarray:
    """fp64 P (batch * m * n): the row softmax of the "nt" product alpha * A_b @ B_b^T, each of
    the batch * m rows normalised over its n values (Section 6's score product, then Section
    2's softmax). Composed from batched_gemm and the fp64 softmax oracle; k == 0 gives 1/n."""
    from .softmax import softmax as softmax_oracle

    C = batched_gemm(a, b, batch, m, n, k, "nt", alpha, dtype)
    if batch == 0 or m == 0 or n == 0:
        return C
    offsets = np.arange(batch, dtype=np.int64) * (m * n)
    return softmax_oracle(C, "f64", offsets, np.full(batch, m, np.int32), np.full(batch, n, np.int32))
