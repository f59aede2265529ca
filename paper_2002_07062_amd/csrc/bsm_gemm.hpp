// Device code of the batched matrix products around the softmax (Section 6's two batch
// matrix multiplications: scores (512 x 64) x (64 x 512) and context (512 x 512) x (512 x 64),
// batch 384), driven by the same host-built work tables as the softmax: the output C_b of
// every batch index is a slice of m rows by n columns, and an item is a run of its rows.
//
//   layout NT:  C_b = alpha A_b B_b^T   (A_b: m x k, B_b: n x k; e.g. Q K^T)
//   layout NN:  C_b = alpha A_b B_b     (A_b: m x k, B_b: k x n; e.g. P V)
//
// bf16 operands, fp32 accumulation on the matrix cores (v_mfma_f32_32x32x16_bf16), fp32 or
// bf16 (round to nearest even) output.  A wave computes 32 output rows at a time, 32 columns
// per MFMA tile, up to four tiles side by side, as the transposed tile D = B_sub A_sub^T:
// the MFMA's row operand is 32 rows of B (NT: contiguous 16-byte loads; NN: gathered down
// B's columns) and its column operand 32 rows of A (contiguous), so each lane ends with four
// consecutive output columns of one output row -- 16-byte stores.  At these shapes the work
// is bound by HBM (the 512 x 512 output, or input), not by the matrix cores.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "bsm.h"

namespace bsm_mm {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

enum { kNT = 0, kNN = 1 };
constexpr int kTileM = 32;   // output rows per wave step
constexpr int kTileN = 32;   // output columns per MFMA tile
constexpr int kTileK = 16;   // reduction depth per MFMA
constexpr int kMaxTiles = 4; // tiles a wave accumulates side by side

struct Shape {
    int m, n, k;
    int64_t a_batch, b_batch, c_batch;  // elements between consecutive batch indices
    float alpha;
    int vec_a, vec_b;  // 16-byte operand loads allowed (k % 8 == 0 / n % 8 == 0 and aligned)
    int vec_c;         // 4-column stores allowed (n % 4 == 0 and aligned)
};

// Eight bf16 of row `row` of a row-major operand with `len` columns, columns c0 .. c0+7;
// zeros when !ok or past len.  The vector form requires len % 8 == 0 and 16-byte alignment;
// its load is unconditional (the caller passes an in-range row, `ok` only selects zeros) so
// that all of a wave's loads are in flight together.
template <bool VEC>
__device__ __forceinline__ bf16x8 row8(const uint16_t* row, int c0, int len, bool ok) {
    if constexpr (VEC) {
        const int cc = c0 < len ? c0 : len - 8;
        u16x8 v = __builtin_nontemporal_load(reinterpret_cast<const u16x8*>(row + cc));
        if (!ok || c0 >= len) v = u16x8{0, 0, 0, 0, 0, 0, 0, 0};
        return __builtin_bit_cast(bf16x8, v);
    } else {
        u16x8 v;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int cc = c0 + e < len ? c0 + e : len - 1;
            const uint16_t x = row[cc];
            v[e] = (ok && c0 + e < len) ? x : static_cast<uint16_t>(0);
        }
        return __builtin_bit_cast(bf16x8, v);
    }
}

// Eight bf16 down column j (an in-range column) of a row-major k x n operand, rows r0 .. r0+7
// (zeros past k or when !ok).
__device__ __forceinline__ bf16x8 col8(const uint16_t* b, int n, int k, int r0, int j, bool ok) {
    u16x8 v;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const int r = r0 + e < k ? r0 + e : k - 1;
        const uint16_t x = b[static_cast<int64_t>(r) * n + j];
        v[e] = (ok && r0 + e < k) ? x : static_cast<uint16_t>(0);
    }
    return __builtin_bit_cast(bf16x8, v);
}

__device__ __forceinline__ unsigned pack_bf16(float a, float b) {
    return __builtin_bit_cast(unsigned, __builtin_convertvector(f32x2{a, b}, bf16x2));
}

// Stores the four values of a lane for output row `row` (valid when row_ok), columns
// j .. j+3 (those below n).
template <bool BF16OUT, bool VECC>
__device__ __forceinline__ void store4(void* c_row, int j, int n, bool row_ok, float v0, float v1,
                                       float v2, float v3) {
    if (!row_ok || j >= n) return;
    if constexpr (BF16OUT) {
        uint16_t* c = static_cast<uint16_t*>(c_row);
        if (VECC && j + 3 < n) {
            __builtin_nontemporal_store(u32x2{pack_bf16(v0, v1), pack_bf16(v2, v3)},
                                        reinterpret_cast<u32x2*>(c + j));
        } else {
            const float v[4] = {v0, v1, v2, v3};
            for (int e = 0; e < 4 && j + e < n; ++e)
                c[j + e] = __builtin_bit_cast(uint16_t, static_cast<__bf16>(v[e]));
        }
    } else {
        float* c = static_cast<float*>(c_row);
        if (VECC && j + 3 < n) {
            __builtin_nontemporal_store(f32x4{v0, v1, v2, v3}, reinterpret_cast<f32x4*>(c + j));
        } else {
            const float v[4] = {v0, v1, v2, v3};
            for (int e = 0; e < 4 && j + e < n; ++e) c[j + e] = v[e];
        }
    }
}

// Output rows [i0, i0 + rows) (rows <= 32) of batch b: all n columns, tiles of 32 columns,
// up to kMaxTiles at a time sharing each load of A.
template <int LAYOUT, bool BF16OUT, bool VECA, bool VECB, bool VECC>
__device__ __forceinline__ void rows32(const uint16_t* a, const uint16_t* b, void* c,
                                       const Shape& s, int64_t bidx, int i0, int rows, int lane) {
    const int li = lane & 31;  // this lane's output row within the chunk (column operand)
    const int h = lane >> 5;   // which 8 of the 16 reduction indices this lane carries
    const bool row_ok = li < rows;
    const int li_in = row_ok ? li : rows - 1;  // loads stay inside the item's rows
    const uint16_t* a_row = a + bidx * s.a_batch + static_cast<int64_t>(i0 + li_in) * s.k;
    const uint16_t* bb = b + bidx * s.b_batch;
    const int ntiles = (s.n + kTileN - 1) / kTileN;
    char* c_row = static_cast<char*>(c) +
                  (bidx * s.c_batch + static_cast<int64_t>(i0 + li_in) * s.n) * (BF16OUT ? 2 : 4);
    for (int t0 = 0; t0 < ntiles; t0 += kMaxTiles) {
        const int nt = ntiles - t0 < kMaxTiles ? ntiles - t0 : kMaxTiles;  // wave-uniform
        f32x16 acc[kMaxTiles];
#pragma unroll
        for (int t = 0; t < kMaxTiles; ++t) acc[t] = f32x16{};
        for (int k0 = 0; k0 < s.k; k0 += kTileK) {
            const int kk = k0 + 8 * h;
            const bf16x8 av = row8<VECA>(a_row, kk, s.k, row_ok);
#pragma unroll
            for (int t = 0; t < kMaxTiles; ++t) {
                if (t < nt) {
                    const int j = (t0 + t) * kTileN + li;  // this lane's row of the row operand
                    const int jc = j < s.n ? j : s.n - 1;
                    bf16x8 bv;
                    if constexpr (LAYOUT == kNT)
                        bv = row8<VECB>(bb + static_cast<int64_t>(jc) * s.k, kk, s.k, j < s.n);
                    else
                        bv = col8(bb, s.n, s.k, kk, jc, j < s.n);
                    acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bv, av, acc[t], 0, 0, 0);
                }
            }
        }
        // D[jj][ii]: lane (ii = li, h) holds columns jj = 8 g + 4 h + 0..3 of tile t
#pragma unroll
        for (int t = 0; t < kMaxTiles; ++t) {
            if (t < nt) {
                const int jbase = (t0 + t) * kTileN;
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int j = jbase + 8 * g + 4 * h;
                    store4<BF16OUT, VECC>(c_row, j, s.n, row_ok, s.alpha * acc[t][4 * g],
                                          s.alpha * acc[t][4 * g + 1], s.alpha * acc[t][4 * g + 2],
                                          s.alpha * acc[t][4 * g + 3]);
                }
            }
        }
    }
}

// Worker loop: worker v (a workgroup, or one wave when per_wave) runs its items; an item's
// rows are taken 32 at a time (split where a batch ends), the workgroup's waves splitting
// them when they share the item.
template <int LAYOUT, bool BF16OUT, bool VECA, bool VECB, bool VECC>
__device__ __forceinline__ void gemm_worker(const uint16_t* a, const uint16_t* b, void* c,
                                            const Shape& s, const int32_t* __restrict__ worker_ptr,
                                            const bsm_item* __restrict__ items, int per_wave,
                                            bsm_trace_rec* __restrict__ trace) {
    const int w = blockIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
    const int nwaves = static_cast<int>(blockDim.x) >> 6;
    const int lane = static_cast<int>(threadIdx.x) & 63;
    const uint64_t t0 = trace ? __builtin_amdgcn_s_memrealtime() : 0;
    const int worker = per_wave ? w * nwaves + wave : w;
    const int my_wave = per_wave ? 0 : wave;
    const int my_nwaves = per_wave ? 1 : nwaves;
    uint32_t done = 0;
    const int i_begin = worker_ptr[worker];
    const int i_end = worker_ptr[worker + 1];
    for (int it = i_begin; it < i_end; ++it) {
        const int64_t e0 = items[it].elem_offset;
        const int nrows = items[it].nrows;
        const int reps = items[it].reps;
        const int64_t stride = static_cast<int64_t>(items[it].rep_stride) * s.n;
        for (int r = 0; r < reps; ++r) {
            // Output rows are numbered batch after batch (row G = b m + i); a run may cross
            // from one batch into the next, so each 32-row chunk is split at batch ends.
            const int64_t g0 = (e0 + r * stride) / s.n;
            for (int q = my_wave * kTileM; q < nrows; q += my_nwaves * kTileM) {
                int64_t g = g0 + q;
                int left = nrows - q < kTileM ? nrows - q : kTileM;
                while (left > 0) {
                    const int64_t bidx = g / s.m;
                    const int i = static_cast<int>(g - bidx * s.m);
                    const int seg = s.m - i < left ? s.m - i : left;
                    rows32<LAYOUT, BF16OUT, VECA, VECB, VECC>(a, b, c, s, bidx, i, seg, lane);
                    done += static_cast<uint32_t>(seg);
                    g += seg;
                    left -= seg;
                }
            }
        }
    }
    if (trace && lane == 0) {
        bsm_trace_rec rec;
        rec.wg = static_cast<uint32_t>(w);
        rec.xcc_id = __builtin_amdgcn_s_getreg(20 | (0 << 6) | ((4 - 1) << 11)) & 0xF;
        rec.hw_id = __builtin_amdgcn_s_getreg(4 | (0 << 6) | ((32 - 1) << 11));
        rec.rows = done;
        rec.t_start = t0;
        rec.t_end = __builtin_amdgcn_s_memrealtime();
        trace[static_cast<int64_t>(w) * nwaves + wave] = rec;
    }
}

template <int LAYOUT, bool BF16OUT, bool VECA, bool VECB, bool VECC>
__global__ void __launch_bounds__(1024)
bsm_gemm_kernel(const uint16_t* a, const uint16_t* b, void* c, Shape s,
                const int32_t* __restrict__ worker_ptr, const bsm_item* __restrict__ items,
                int per_wave, bsm_trace_rec* __restrict__ trace) {
    gemm_worker<LAYOUT, BF16OUT, VECA, VECB, VECC>(a, b, c, s, worker_ptr, items, per_wave, trace);
}

}  // namespace bsm_mm
