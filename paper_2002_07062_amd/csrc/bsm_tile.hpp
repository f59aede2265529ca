// Register-tile rule shared by the kernel (which executes it) and the planner (which sizes
// work pieces to whole tile steps).  constexpr functions are usable from host and device.
#pragma once

#include <cstdint>

namespace bsm {

constexpr int kWave = 64;
constexpr int kVecBytes = 16;   // one 128-bit access

// Register tile of an aligned row of `nvec` 16-byte vectors in a kernel of class `kclass`: G
// lanes per row (a group), V vectors per lane, U rows per group in flight, 64 / G groups per
// wave.  V = 0: beyond the register tiles of the class.
//
// Measured on MI355X (uniform batches of ~200 MB): a tile streams at the copy rate when it is
// full; a partly filled one loses in proportion to the bytes its lanes keep in flight.  fp32
// rows (8 waves per CU) therefore take tiles that keep about 4-5 KiB per wave in flight: more
// rows per group for half-filled 32-lane tiles, 5 vectors per lane where a 5-vector tile fits
// the row better than a power of two.  bf16 rows run 16 waves per CU with twice the arithmetic
// per byte: larger tiles raise their registers past that occupancy, and they keep the
// power-of-two tiles with four 16-byte loads per lane in flight.  Rows of 33..64 vectors take
// 32 lanes x 2 vectors rather than 64 x 1 (a shorter butterfly and half the per-row work per
// value: +7% on 384 x 512 x 512 bf16).
struct Tile {
    int G;
    int V;
    int U;
};

constexpr Tile tile_for(int64_t nvec, int kclass, int elem_bytes, bool packed = true) {
    // Rows of 5-7, 9-10 and 17-21 vectors in plans of kernel class 0: packed groups of exactly
    // nvec lanes, 64 / nvec rows side by side per wave (G = nvec, not a power of two, marks the
    // packed tile), where a power-of-two group leaves 34-69% of its lanes idle; rows of 8
    // vectors take eight 8-lane groups.  Measured against the tiles they replace (uniform
    // ~200 MB batches, alternating runs on one box, GB/s): fp32 20 2940 -> 5270, 24 3540 ->
    // 5310, 28 3910 -> 5240, 32 4210 -> 5710, 36 4590 -> 5250, 40 4980 -> 5320, 68 4670 ->
    // 4960, 72 5030 -> 5060, 84 5000 -> 5260; bf16 64 4500 -> 5180, 72 4610 -> 5080, 80 equal,
    // 136 4270 -> 4650, 144 4480 -> 4860, 168 4660 -> 5080.  44 and 48 fp32 (5 groups of 11 or
    // 12) lost 2-3%, and so did the ragged batch (-1.5%) with the packed code in its class-2
    // instance even where no row took it, so higher classes keep the power-of-two tiles.  Only
    // rows that start and end on 16-byte vectors (`packed`).
    if (packed && kclass == 0 && ((nvec >= 5 && nvec <= 7) || (nvec >= 9 && nvec <= 10) || (nvec >= 17 && nvec <= 21)))
        return Tile{static_cast<int>(nvec), 1, 4};
    if (kclass == 0 && nvec == 8) return Tile{8, 1, 4};
    if (nvec <= 16) return Tile{16, 1, 4};
    if (elem_bytes == 4 && nvec <= 24) return Tile{32, 1, 8};
    if (nvec <= 32) return Tile{32, 1, 4};
    if (kclass >= 1) {
        if (elem_bytes == 4) {
            if (nvec <= 40) return Tile{32, 2, 4};
            if (nvec <= 64) return Tile{32, 2, 2};
            if (nvec <= 80) return Tile{16, 5, 1};
            if (nvec <= 96) return Tile{64, 2, 3};
        }
        if (nvec <= 64) return Tile{32, 2, 2};
        if (nvec <= 128) return Tile{64, 2, 2};
    }
    if (kclass >= 2) {
        if (elem_bytes == 4 && nvec <= 160) return Tile{32, 5, 1};
        if (nvec <= 256) return Tile{64, 4, 1};
    }
    if (kclass >= 3) {
        if (elem_bytes == 4 && nvec <= 320) return Tile{64, 5, 1};
        if (nvec <= 512) return Tile{64, 8, 1};
    }
    if (kclass >= 4) {
        // long-row plans (workgroup workers, 8 waves per CU): rows of up to 768 vectors are
        // still held by one wave each, the workgroup's waves taking turns at the item's rows
        // (a 16-vector tile measured 3.5% slower than the workgroup-held row at 1024 fp32
        // vectors, and does not fit 256 registers in bf16)
        if (nvec <= 640) return Tile{64, 10, 1};
        if (nvec <= 768) return Tile{64, 12, 1};
    }
    return Tile{64, 0, 1};
}

// Register tile of the backward pass (two input streams, y and dy) for an aligned row of
// `nvec` vectors; V = 0: the one-wave or workgroup paths.  bf16 rows keep half the forward
// pass's rows in flight.  fp32 rows, like the forward pass, keep about 4-5 KiB of both streams
// per wave in flight where a power-of-two tile is partly empty, and rows of 257-512 vectors
// keep a 64 x 8 register tile (the one-wave path, staging y and dy in LDS, ran them at
// 3.7 TB/s).
constexpr Tile tile_for_bwd(int64_t nvec, int kclass, int elem_bytes, bool packed = true) {
    const bool f = elem_bytes == 4;
    // plans of kernel class 0: rows of 5-7 vectors (fp32 also 9-10 and 17-21) in packed
    // groups, of 8 in 8-lane groups, as in the forward pass (bf16 rows of 9 and 18 vectors lost
    // 3% packed: their 16- and 32-lane tiles already keep twice the elements per lane busy)
    if (packed && kclass == 0 &&
        ((nvec >= 5 && nvec <= 7) || (f && ((nvec >= 9 && nvec <= 10) || (nvec >= 17 && nvec <= 21)))))
        return Tile{static_cast<int>(nvec), 1, 2};
    if (kclass == 0 && nvec == 8) return Tile{8, 1, 2};
    if (nvec <= 16) return Tile{16, 1, 2};
    if (f && nvec <= 24) return Tile{32, 1, 4};
    if (nvec <= 32) return Tile{32, 1, 2};
    if (kclass >= 1) {
        if (f && nvec <= 40) return Tile{64, 1, 4};
        if (nvec <= 64) return Tile{64, 1, 2};
        if (f && nvec <= 80) return Tile{64, 2, 2};
        if (nvec <= 128) return Tile{64, 2, 1};
    }
    if (kclass >= 2 && nvec <= 256) return Tile{64, 4, 1};
    if (f && kclass >= 3 && nvec <= 512) return Tile{64, 8, 1};
    return Tile{64, 0, 1};
}

// Rows beyond the register tile are held in the registers of a whole workgroup: kTeamThreads
// threads with up to kTeamValues values per lane in kernel class 4 (rows of up to
// kTeamThreads * kTeamValues elements), twice that in class 5, whose instances need twice the
// registers, and in class 6 (longer rows) workgroups of 2 * kTeamThreads threads with twice
// the values, one workgroup per CU.
constexpr int kTeamThreads = 256;
constexpr int kTeamValues = 32;
constexpr int kLongestClass = 6;
// Threads of the workgroup that holds a row, by kernel class (>= 4).
constexpr int team_threads(int kernel_class) {
    return kernel_class >= kLongestClass ? 2 * kTeamThreads : kTeamThreads;
}

// Rows a workgroup holds at a time (kernel class >= 4) when a row takes `per_lane` vectors per
// lane: two for the shortest rows (at most 3 vectors per lane) and for bf16 rows of 5 or 6
// vectors per lane in classes 5 and 6, one otherwise (the kernel's team_item makes the same
// choice).
constexpr int team_rows_in_flight(int per_lane, int kernel_class, int elem_bytes) {
    const int max_l = (kernel_class >= 5 ? 2 : 1) * kTeamValues * elem_bytes / kVecBytes;
    return (per_lane <= 3 || (elem_bytes == 2 && max_l >= 6 && per_lane <= 6)) ? 2 : 1;
}

// Rows one worker finishes per step for a row of `cols` elements (aligned rows): one wave's
// tile step, times the waves of the workgroup that is the worker in long-row plans (kernel
// class >= 4); for a row the workgroup holds, the rows it holds at a time, so that a piece of
// a balanced table does not leave half of a row pair empty.
constexpr int wave_step_rows(int64_t cols, int elem_bytes, int kernel_class) {
    const int64_t nvec = (cols * elem_bytes + kVecBytes - 1) / kVecBytes;
    const Tile t = tile_for(nvec, kernel_class, elem_bytes);
    if (t.V == 0) {
        if (kernel_class < 4) return 1;
        const int nt = team_threads(kernel_class);
        return team_rows_in_flight(static_cast<int>((nvec + nt - 1) / nt), kernel_class, elem_bytes);
    }
    const int rows = (kWave / t.G) * t.U;
    return kernel_class >= 4 ? rows * (team_threads(kernel_class) / kWave) : rows;
}

}  // namespace bsm
