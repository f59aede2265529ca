"""Seeded random slice geometries for the randomized planner and parity tests: slices in a
random order with random gaps (in half the geometries every slice start and row length a
multiple of 8 elements, so aligned paths run), empty slices, widths across every
register-tile class and long rows of both long-row kernel classes. Input generation only (no softmax arithmetic)."""

import numpy as np

import workloads

WIDTHS = [1, 3, 7, 8, 15, 16, 17, 31, 33, 64, 72, 100, 128, 129, 200, 256, 260, 511, 512, 513,
          700, 1000, 1024, 1100, 2048, 2051, 3000, 4096, 5000, 8192, 9000, 12000, 16384, 20000]


def geometry(seed: int, max_batch: int = 40, max_rows: int = 120, dtype: str = "f32",
             long_rows: bool = True) -> workloads.Workload:
    rng = np.random.default_rng(seed)
    batch = int(rng.integers(0, max_batch + 1))
    widths = WIDTHS if long_rows else [c for c in WIDTHS if c <= 2048]
    cols = rng.choice(widths, size=batch).astype(np.int32)
    rows = rng.integers(0, max_rows + 1, size=batch).astype(np.int32)
    rows[rng.random(batch) < 0.1] = 0  # some empty slices
    base = int(rng.integers(0, 40))
    gaps = rng.integers(0, 50, size=batch)
    if rng.random() < 0.5:  # every slice start 16-byte aligned (for fp32 and bf16)
        base, gaps = 8 * base, 8 * gaps
        cols = np.where(cols % 8 == 0, cols, cols - cols % 8 + 8).astype(np.int32)
    order = rng.permutation(batch)
    offsets = np.zeros(batch + 1, dtype=np.int64)
    pos = base
    for s in order:  # slices laid out in a random order
        offsets[s] = pos
        pos += int(rows[s]) * int(cols[s]) + int(gaps[s])
    offsets[batch] = pos
    x = (rng.standard_normal(pos, dtype=np.float32) * np.float32(3.0))
    if dtype == "bf16":
        x = workloads._to_bf16_bits(x)
    return workloads.Workload(f"random_{seed}", dtype, x, offsets, rows, cols, uniform=False)


def topology(seed: int) -> dict:
    rng = np.random.default_rng(10_000 + seed)
    n_xcd = int(rng.choice([1, 2, 3, 8]))
    n_cu = n_xcd * int(rng.choice([1, 2, 5, 32]))
    return dict(n_cu=n_cu, n_xcd=n_xcd, wg_per_cu=int(rng.choice([1, 2, 3])),
                wg_threads=int(rng.choice([64, 128, 256, 512])))
