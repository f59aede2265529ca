// Register-tile rule shared by the kernel (which executes it) and the planner (which sizes
// work pieces to whole tile steps).  constexpr functions are usable from host and device.
#pragma once

#include <cstdint>

namespace bsm {

constexpr int kWave = 64;
constexpr int kVecBytes = 16;   // one 128-bit access
constexpr int kVecsInFlight = 4;  // 16-byte loads per lane a wave keeps in flight (any dtype)

// Lanes per row G and 16-byte vectors per lane V for a row of `nvec` vectors.  Rows beyond
// 64 * max_v vectors take the two-pass path (G = 64, V = 0).
struct Tile {
    int G;
    int V;
};

constexpr Tile tile_for(int64_t nvec, int max_v) {
    if (nvec <= 16) return Tile{16, 1};
    if (nvec <= 32) return Tile{32, 1};
    if (max_v >= 2 && nvec <= 64) return Tile{32, 2};  // (kernel class >= 1 for such rows)
    if (nvec <= 64) return Tile{64, 1};
    if (max_v >= 2 && nvec <= 128) return Tile{64, 2};
    if (max_v >= 4 && nvec <= 256) return Tile{64, 4};
    if (max_v >= 8 && nvec <= 512) return Tile{64, 8};
    return Tile{64, 0};
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

// Rows per group a wave keeps in flight: enough rows that each lane has kVecsInFlight 16-byte
// loads outstanding (one row for the element-wise and two-pass paths).
constexpr int rows_per_group_in_flight(int V, bool vec_path) {
    return (!vec_path || V == 0 || V >= kVecsInFlight) ? 1 : kVecsInFlight / V;
}

// Rows a wave keeps in flight per step: that many rows per group of G lanes, 64/G groups.
constexpr int rows_in_flight(int G, int V, bool vec_path) {
    return (kWave / G) * rows_per_group_in_flight(V, vec_path);
}

// Largest register tile (vectors per lane) a kernel class carries.
constexpr int max_v_of_class(int kernel_class) {
    return kernel_class <= 0 ? 1 : kernel_class == 1 ? 2 : kernel_class == 2 ? 4 : 8;
}

// Rows one wave finishes per step for a row of `cols` elements (aligned rows).
constexpr int wave_step_rows(int64_t cols, int elem_bytes, int kernel_class) {
    const int64_t nvec = (cols * elem_bytes + kVecBytes - 1) / kVecBytes;
    const Tile t = tile_for(nvec, max_v_of_class(kernel_class));
    return rows_in_flight(t.G, t.V, true);
}

}  // namespace bsm
