"""Seeded synthetic inputs for the batched row softmax.

This module only draws inputs: slice geometry (rows, cols, packed element offsets) and values.
It holds none of the softmax arithmetic and none of the scheduling logic, so that the fp64
oracle under ``oracle/`` and the HIP path can both be fed from it without sharing code.

Workloads follow the paper's problem statement (Section 2): B small 2-D slices packed along
rows into one (B*R) x C tensor, as in BERT's 384 attention-score slices of 512 x 512. There is
no public dataset behind them; N(0, sigma^2) values stand in for scaled q.k/sqrt(d_k) scores.

Draw order per workload: geometry first (mask lengths, or slice rows then slice cols), then
values, so geometry and data are reproducible separately.
"""

from __future__ import annotations

import dataclasses

import numpy as np

F32 = "f32"
BF16 = "bf16"

BF16_NEG_INF = np.uint16(0xFF80)


@dataclasses.dataclass(frozen=True)
class Spec:
    name: str
    batch: int
    rows: int  # uniform R (0 for ragged)
    cols: int  # uniform C (0 for ragged)
    dtype: str
    sigma: float
    seed: int
    mask_max: int = -1  # >= 0: per-slice key-padding length L ~ U{0..mask_max}
    ragged: tuple | None = None  # (lo, hi, step): R and C drawn from {lo, lo+step, .., hi}
    doc: str = ""


SPECS = {
    "c1_8x64x64_f32": Spec(
        "c1_8x64x64_f32", 8, 64, 64, F32, 1.0, 1,
        doc="8 slices x 64x64 fp32 packed as 512x64, N(0,1)"),
    "c2_384x512x512_f32": Spec(
        "c2_384x512x512_f32", 384, 512, 512, F32, 3.0, 2,
        doc="384 slices x 512x512 fp32 packed as 196608x512, N(0,9): BERT attention scores"),
    "c3_384x512x512_bf16_mask": Spec(
        "c3_384x512x512_bf16_mask", 384, 512, 512, BF16, 3.0, 3, mask_max=448,
        doc="384 x 512x512 bf16, N(0,9), last L_s columns of slice s set to -inf, "
            "L_s ~ U{0..448}"),
    "c4_16384x128x128_f32": Spec(
        "c4_16384x128x128_f32", 16384, 128, 128, F32, 2.0, 4,
        doc="16384 slices x 128x128 fp32, N(0,4): many tiny slices"),
    "c5_384_ragged_f32": Spec(
        "c5_384_ragged_f32", 384, 0, 0, F32, 3.0, 5, ragged=(64, 1024, 8),
        doc="384 ragged fp32 slices, R_s and C_s independently uniform over multiples of 8 "
            "in [64, 1024], packed contiguously with int64 offsets, N(0,9)"),
    # long rows (beyond the register tile): long-context attention scores
    "long_128x64x4096_f32": Spec(
        "long_128x64x4096_f32", 128, 64, 4096, F32, 3.0, 7,
        doc="128 slices x 64x4096 fp32, N(0,9): 4 vectors per lane of a 256-thread workgroup"),
    "long_64x64x8192_f32": Spec(
        "long_64x64x8192_f32", 64, 64, 8192, F32, 3.0, 6,
        doc="64 slices x 64x8192 fp32, N(0,9): the longest rows of kernel class 4 (8 vectors per lane)"),
    # rows that do not start or end on a 16-byte vector (shifted rows)
    "odd_64x768x1001_f32": Spec(
        "odd_64x768x1001_f32", 64, 768, 1001, F32, 3.0, 9,
        doc="64 slices x 768x1001 fp32, N(0,9): every row starts at a different phase of the "
            "16-byte vectors"),
    "long_16x64x32768_f32": Spec(
        "long_16x64x32768_f32", 16, 64, 32768, F32, 3.0, 10,
        doc="16 slices x 64x32768 fp32, N(0,9): rows held by a 512-thread workgroup (class 6)"),
    "long_32x64x16384_f32": Spec(
        "long_32x64x16384_f32", 32, 64, 16384, F32, 3.0, 8,
        doc="32 slices x 64x16384 fp32, N(0,9): the longest register-held rows (class 5, 16 vectors per lane)"),
    # bf16 rows just past the one-wave register tile: 513 and 1025 16-byte vectors
    "long_128x96x4104_bf16": Spec(
        "long_128x96x4104_bf16", 128, 96, 4104, BF16, 3.0, 11,
        doc="128 slices x 96x4104 bf16, N(0,9): 513 vectors per row, one past the 512 of the "
            "largest short-row tile"),
    "long_64x96x8200_bf16": Spec(
        "long_64x96x8200_bf16", 64, 96, 8200, BF16, 3.0, 12,
        doc="64 slices x 96x8200 bf16, N(0,9): 1025 vectors per row, held by a workgroup"),
}
# Uniform fp32 batches of ~200 MB input at one row width each: full and partly filled register
# tiles (the widths of the ragged workload run from 64 to 1024).
for _c in (64, 72, 96, 136, 264, 520):
    _r = round(50e6 / (64 * _c))
    _n = f"width_64x{_r}x{_c}_f32"
    SPECS[_n] = Spec(_n, 64, _r, _c, F32, 3.0, 100 + _c,
                     doc=f"64 slices x {_r}x{_c} fp32, N(0,9): rows of {_c // 4} 16-byte vectors")

# Short aliases used by the bench and the tests.
ALIASES = {"c1": "c1_8x64x64_f32", "c2": "c2_384x512x512_f32",
           "c3": "c3_384x512x512_bf16_mask", "c4": "c4_16384x128x128_f32",
           "c5": "c5_384_ragged_f32", "long": "long_64x64x8192_f32",
           "long4k": "long_128x64x4096_f32", "long16k": "long_32x64x16384_f32",
           "odd": "odd_64x768x1001_f32", "long32k": "long_16x64x32768_f32",
           "long4104bf16": "long_128x96x4104_bf16", "long8200bf16": "long_64x96x8200_bf16"}
ALIASES.update({f"w{s.cols}": n for n, s in SPECS.items() if n.startswith("width_")})


@dataclasses.dataclass
class Workload:
    name: str
    dtype: str
    x: np.ndarray  # flat: float32, or uint16 holding bf16 bit patterns
    offsets: np.ndarray  # int64 [batch + 1], element offsets of each slice
    rows: np.ndarray  # int32 [batch]
    cols: np.ndarray  # int32 [batch]
    uniform: bool
    mask_len: np.ndarray | None = None  # int32 [batch] for masked workloads

    @property
    def batch(self) -> int:
        return int(self.rows.shape[0])

    @property
    def elem_size(self) -> int:
        return 4 if self.dtype == F32 else 2

    @property
    def n_elements(self) -> int:
        return int(np.sum(self.rows.astype(np.int64) * self.cols.astype(np.int64)))

    @property
    def algorithmic_bytes(self) -> int:
        """Every input element read once plus every output element written once."""
        return 2 * self.n_elements * self.elem_size


def spec(name: str) -> Spec:
    return SPECS[ALIASES.get(name, name)]


def _to_bf16_bits(x: np.ndarray) -> np.ndarray:
    # Round-to-nearest-even fp32 -> bf16 via torch's CPU conversion (input preparation only).
    import torch

    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def packed_offsets(rows: np.ndarray, cols: np.ndarray) -> np.ndarray:
    """Contiguous packing: slice s starts where slice s-1 ends."""
    sizes = rows.astype(np.int64) * cols.astype(np.int64)
    off = np.zeros(rows.shape[0] + 1, dtype=np.int64)
    np.cumsum(sizes, out=off[1:])
    return off


def generate(name: str, seed: int | None = None, batch: int | None = None,
             values: bool = True) -> Workload:
    """Draw one workload. `batch` (<= the spec's) keeps only the first slices' geometry, with
    the same draws for them, for tests that need a small but faithful sample. values=False
    draws the geometry only (x is empty)."""
    sp = spec(name)
    rng = np.random.default_rng(sp.seed if seed is None else seed)
    B = sp.batch
    mask_len = None
    if sp.ragged is not None:
        lo, hi, step = sp.ragged
        n = (hi - lo) // step + 1
        rows = (lo + step * rng.integers(0, n, size=B)).astype(np.int32)
        cols = (lo + step * rng.integers(0, n, size=B)).astype(np.int32)
    else:
        rows = np.full(B, sp.rows, dtype=np.int32)
        cols = np.full(B, sp.cols, dtype=np.int32)
        if sp.mask_max >= 0:
            mask_len = rng.integers(0, sp.mask_max + 1, size=B).astype(np.int32)
    if batch is not None:
        if not 0 <= batch <= B:
            raise ValueError(f"batch {batch} outside [0, {B}]")
        rows, cols = rows[:batch], cols[:batch]
        if mask_len is not None:
            mask_len = mask_len[:batch]
    offsets = packed_offsets(rows, cols)
    total = int(offsets[-1])
    if not values:
        return Workload(sp.name, sp.dtype, np.zeros(0, np.float32), offsets, rows, cols,
                        uniform=sp.ragged is None, mask_len=mask_len)
    x = rng.standard_normal(total, dtype=np.float32)
    x *= np.float32(sp.sigma)
    if sp.dtype == BF16:
        x = _to_bf16_bits(x)
        if mask_len is not None:
            R, C = int(rows[0]) if len(rows) else 0, int(cols[0]) if len(cols) else 0
            v = x.reshape(-1, R, C) if total else x.reshape(0, max(R, 1), max(C, 1))
            for s, L in enumerate(mask_len):
                if L:
                    v[s, :, C - L:] = BF16_NEG_INF
    return Workload(sp.name, sp.dtype, x, offsets, rows, cols,
                    uniform=sp.ragged is None, mask_len=mask_len)


def custom(rows, cols, dtype=F32, sigma=1.0, seed=0, gap=0, base=0) -> Workload:
    """Arbitrary ragged geometry for edge-case tests: slice s has rows[s] x cols[s] elements,
    packed in order with `gap` spare elements after each slice and `base` before the first."""
    rows = np.asarray(rows, dtype=np.int32)
    cols = np.asarray(cols, dtype=np.int32)
    sizes = rows.astype(np.int64) * cols.astype(np.int64) + gap
    offsets = np.zeros(rows.shape[0] + 1, dtype=np.int64)
    offsets[0] = base
    np.cumsum(sizes, out=offsets[1:])
    offsets[1:] += base
    total = int(offsets[-1])
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(total, dtype=np.float32) * np.float32(sigma)
    if dtype == BF16:
        x = _to_bf16_bits(x)
    return Workload("custom", dtype, x, offsets, rows, cols, uniform=False)


def gradient(w: Workload, seed: int = 1000) -> np.ndarray:
    """Upstream gradient dy for the backward pass of workload `w`: N(0, 1) at every element of
    `w.x` (gaps included; their values never affect dx), in w's dtype (bf16 as raw bit patterns, rounded to
    nearest even). Drawn from its own seed so the forward inputs are unaffected."""
    rng = np.random.default_rng(seed)
    g = rng.standard_normal(w.x.shape[0], dtype=np.float32)
    return _to_bf16_bits(g) if w.dtype == BF16 else g
