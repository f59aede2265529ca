// Device code of the batched matrix products around the softmax (Section 6's two batch
// matrix multiplications: scores (512 x 64) x (64 x 512) and context (512 x 512) x (512 x 64),
// batch 384), driven by the same host-built work tables as the softmax: the output C_b of
// every batch index is a slice of m rows by n columns, and an item is a run of its rows.
//
//   layout NT:  C_b = alpha A_b B_b^T   (A_b: m x k, B_b: n x k; e.g. Q K^T)
//   layout NN:  C_b = alpha A_b B_b     (A_b: m x k, B_b: k x n; e.g. P V)
//
// bf16 operands, fp32 accumulation on the matrix cores (v_mfma_f32_32x32x16_bf16), fp32 or
// bf16 (round to nearest even) output.  A wave computes 32 output rows at a time in blocks of
// 64 columns (two 32 x 32 MFMA tiles), as the transposed tile D = B_sub A_sub^T so that each
// lane ends with four consecutive output columns.  Operands are staged in the wave's LDS from
// 16-byte loads (NN's B transposed on the way in), one step ahead: a step's loads are in
// flight while the previous step computes; the output block goes through LDS too and is
// stored as whole rows.  At these shapes the work is bound by HBM (the 512 x 512 output, or
// input), not by the matrix cores.
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
constexpr int kMaxTiles = 2; // tiles a wave accumulates side by side

struct Shape {
    int m, n, k;
    int64_t a_batch, b_batch, c_batch;  // elements between consecutive batch indices
    float alpha;
};

// One step of a wave's work on a 32-row chunk: the output column block [j0, j0 + 64) (two
// 32 x 32 MFMA tiles) and the reduction slice [k0, k0 + 64).  Per-wave LDS layout (bf16
// elements): A block [32][kLdk], B block [64][kLdk] (B's rows for NT, B's columns for NN: the
// MFMA's row operand either way), rows padded so that a ds_read_b128 of 32 rows spreads over
// the banks.  After a column block's last step the output block is staged in the same region
// as [32][kLdc] fp32 and stored as whole rows.
constexpr int kChunkK = 64;                 // reduction indices per step
constexpr int kLdk = kChunkK + 8;           // padded LDS row, elements
constexpr int kBlockN = 64;                 // output columns per block (two tiles)
constexpr int kBlockTiles = kBlockN / kTileN;
constexpr int kLdc = kBlockN + 4;           // padded LDS row of the staged output, floats
constexpr int kLdh = kBlockN + 8;           // ... staged as bf16, elements
constexpr int kLdv = kBlockN + 8;           // padded LDS row of NN's B (rows = reduction index)
constexpr int kLdsBytes = (kTileM * kLdc * 4 > (kTileM + kBlockN) * kLdk * 2)
                              ? kTileM * kLdc * 4 : (kTileM + kBlockN) * kLdk * 2;
static_assert(kChunkK * kLdv <= kBlockN * kLdk, "NN's B fits the B region");
constexpr int kAPieces = kTileM * kChunkK / 8 / 64;   // 16-byte pieces of A per lane per step
constexpr int kBPieces = kBlockN * kChunkK / 8 / 64;  // ... of B

__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ unsigned pack_bf16(float a, float b) {
    return __builtin_bit_cast(unsigned, __builtin_convertvector(f32x2{a, b}, bf16x2));
}

// Eight consecutive bf16 of a row-major operand row (`len` columns) from column c, or from
// the row's last whole piece when c is past the row (the caller zeroes such pieces when it
// writes them to LDS).  VEC: one unconditional 16-byte load (len % 8 == 0, 16-byte aligned
// rows), so that no branch or select on the loaded data sits between a step's loads and the
// wait before their use; the scalar form (any len) loads element by element.  Ordinary
// (cache-resident) loads: B is re-read by every row chunk of its batch, A by every column
// block.
template <bool VEC>
__device__ __forceinline__ u16x8 load8(const uint16_t* row, int c, int len) {
    if constexpr (VEC) {
        return *reinterpret_cast<const u16x8*>(row + (c < len ? c : len - 8));
    } else {
        u16x8 v;
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = row[c + e < len ? c + e : len - 1];
        return v;
    }
}

// Zeroes the elements of a piece loaded from columns [c, c + 8) that lie past `len`, or all
// of them when !ok.  VEC (len % 8 == 0, c % 8 == 0): the piece is wholly in or wholly out,
// four 32-bit selects.
template <bool VEC>
__device__ __forceinline__ u16x8 keep8(u16x8 v, int c, int len, bool ok) {
    if constexpr (VEC) {
        const bool in = ok && c < len;
        u32x4 w = __builtin_bit_cast(u32x4, v);
#pragma unroll
        for (int e = 0; e < 4; ++e) w[e] = in ? w[e] : 0u;
        return __builtin_bit_cast(u16x8, w);
    } else {
        u16x8 z;
#pragma unroll
        for (int e = 0; e < 8; ++e) z[e] = (ok && c + e < len) ? v[e] : static_cast<unsigned short>(0);
        return z;
    }
}

// The operand pieces of one step, held in registers between their loads and their LDS writes
// so that a step's loads are in flight while earlier steps compute.
struct Pieces {
    u16x8 a[kAPieces];
    u16x8 b[kBPieces];
};

// Piece q of a lane.  A and NT's B: lanes walk rows 8 pieces (128 bytes) at a time.  NN's B:
// lane = reduction index, piece q = columns 8q .. 8q+7, so that the transposed LDS writes of
// consecutive lanes fall in consecutive bytes.
__device__ __forceinline__ int piece_row(int lane, int q) { return (lane + 64 * q) / (kChunkK / 8); }
__device__ __forceinline__ int piece_col(int lane, int q) { return ((lane + 64 * q) % (kChunkK / 8)) * 8; }
// NN's B: rows of kBlockN columns, kBlockN / 8 pieces each
__device__ __forceinline__ int piece_nn_row(int lane, int q) { return (lane + 64 * q) / (kBlockN / 8); }
__device__ __forceinline__ int piece_nn_col(int lane, int q) { return ((lane + 64 * q) % (kBlockN / 8)) * 8; }

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

// MFMA row operand of NN from row-major B in LDS: lane (li, h) of tile t gets B[kk + 8h + e]
// [32t + li] for e = 0..7.  ds_read_b64_tr_b16 works on groups of 16 lanes: lane i of a group
// receives element i % 4 of the 8-byte loads of the group's lanes 4r + i / 4, r = 0..3; so
// group lane s points at row kb + s / 4, columns jb + 4 (s % 4) .. +3, and lane i ends with
// column jb + i of rows kb .. kb+3.  Two reads (kb and kb + 4) give the eight rows.
__device__ __forceinline__ bf16x8 nn_row_operand(const uint16_t* lb, int t, int kk, int lane) {
    const int g = lane >> 4, sl = lane & 15;
    const int kb = kk + 8 * (g >> 1), jb = t * kTileN + 16 * (g & 1);
    const uint16_t* p0 = lb + (kb + (sl >> 2)) * kLdv + jb + 4 * (sl & 3);
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p0));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p0 + 4 * kLdv));
    u16x8 v;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        v[e] = static_cast<unsigned short>(lo[e]);
        v[e + 4] = static_cast<unsigned short>(hi[e]);
    }
    return __builtin_bit_cast(bf16x8, v);
}

// A's pieces of the reduction slice [k0, k0 + 64) of the wave's rows, and their LDS writes
// (rows past `rows` and columns past k zeroed).
template <bool VEC>
__device__ __forceinline__ void load_a(const uint16_t* a_blk, const Shape& s, int rows, int k0,
                                       int lane, u16x8 (&pa)[kAPieces]) {
#pragma unroll
    for (int q = 0; q < kAPieces; ++q) {
        const int r = piece_row(lane, q);
        pa[q] = load8<VEC>(a_blk + static_cast<int64_t>(r < rows ? r : rows - 1) * s.k,
                           k0 + piece_col(lane, q), s.k);
    }
}

template <bool VEC>
__device__ __forceinline__ void write_a(const u16x8 (&pa)[kAPieces], const Shape& s, int rows,
                                        int k0, int lane, uint16_t* la) {
#pragma unroll
    for (int q = 0; q < kAPieces; ++q) {
        const int r = piece_row(lane, q), c = piece_col(lane, q);
        *reinterpret_cast<u16x8*>(la + r * kLdk + c) = keep8<VEC>(pa[q], k0 + c, s.k, r < rows);
    }
}

template <int LAYOUT, bool VEC, bool WITH_A>
__device__ __forceinline__ void load_step(const uint16_t* a_blk, const uint16_t* b_blk,
                                          const Shape& s, int rows, int j0, int k0, int lane,
                                          Pieces& p) {
    if (s.k == 0) {  // empty reduction: nothing to read (write_step zeroes every piece)
        if constexpr (WITH_A) {
#pragma unroll
            for (int q = 0; q < kAPieces; ++q) p.a[q] = u16x8{0, 0, 0, 0, 0, 0, 0, 0};
        }
#pragma unroll
        for (int q = 0; q < kBPieces; ++q) p.b[q] = u16x8{0, 0, 0, 0, 0, 0, 0, 0};
        return;
    }
    if constexpr (WITH_A) load_a<VEC>(a_blk, s, rows, k0, lane, p.a);
    if constexpr (LAYOUT == kNT) {
#pragma unroll
        for (int q = 0; q < kBPieces; ++q) {
            const int j = j0 + piece_row(lane, q);
            p.b[q] = load8<VEC>(b_blk + static_cast<int64_t>(j < s.n ? j : s.n - 1) * s.k,
                                k0 + piece_col(lane, q), s.k);
        }
    } else {
#pragma unroll
        for (int q = 0; q < kBPieces; ++q) {
            const int kr = k0 + piece_nn_row(lane, q);
            p.b[q] = load8<VEC>(b_blk + static_cast<int64_t>(kr < s.k ? kr : s.k - 1) * s.n,
                                j0 + piece_nn_col(lane, q), s.n);
        }
    }
}

template <int LAYOUT, bool VEC, bool WITH_A>
__device__ __forceinline__ void write_step(const Pieces& p, const Shape& s, int rows, int j0,
                                           int k0, int lane, uint16_t* la, uint16_t* lb) {
    if constexpr (WITH_A) write_a<VEC>(p.a, s, rows, k0, lane, la);
    if constexpr (LAYOUT == kNT) {
#pragma unroll
        for (int q = 0; q < kBPieces; ++q) {
            const int r = piece_row(lane, q), c = piece_col(lane, q);
            *reinterpret_cast<u16x8*>(lb + r * kLdk + c) = keep8<VEC>(p.b[q], k0 + c, s.k, j0 + r < s.n);
        }
    } else {
        // B's rows k0 .. k0+63 as they are (row = reduction index, kLdv elements apart);
        // the MFMA operand is read back transposed (ds_read_b64_tr_b16)
#pragma unroll
        for (int q = 0; q < kBPieces; ++q) {
            const int kr = piece_nn_row(lane, q), c = piece_nn_col(lane, q);
            *reinterpret_cast<u16x8*>(lb + kr * kLdv + c) =
                keep8<VEC>(p.b[q], j0 + c, s.n, k0 + kr < s.k);
        }
    }
}

// Stores the staged output block (rows [i0, i0 + rows), columns [j0, j0 + jn) of batch b)
// as whole rows: 16 lanes x 4 columns per row, four rows per store instruction.
// Stores a staged output block (rows [i0, i0 + rows), columns [j0, j0 + jn)) as whole rows:
// 16 lanes x 4 fp32 columns, four rows per instruction.
template <bool VEC>
__device__ __forceinline__ void store_block_f32(float* c, const Shape& s, int64_t bidx, int i0, int rows,
                                            int j0, int jn, int lane, const float* lc) {
    const int col = (lane & 15) * 4;
    const int rq = lane >> 4;
    // one 64-bit base per lane, advanced by 4 output rows per instruction
    const int64_t off0 = bidx * s.c_batch + static_cast<int64_t>(i0 + rq) * s.n + j0 + col;
    const int64_t step = 4 * static_cast<int64_t>(s.n);
    const bool col_ok = col < jn;
    const bool whole = VEC && col + 3 < jn;
#pragma unroll
    for (int r0 = 0; r0 < kTileM; r0 += 4) {
        const int r = r0 + rq;
        if (r < rows && col_ok) {
            const f32x4 v = *reinterpret_cast<const f32x4*>(lc + r * kLdc + col);
            float* cp = c + off0 + (r0 / 4) * step;
            if (whole) {
                __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(cp));
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (col + e < jn) cp[e] = v[e];
            }
        }
    }
}

// The same for a block staged as bf16 ([32][kLdh]): 8 lanes x 8 columns, eight rows per
// instruction.
template <bool VEC>
__device__ __forceinline__ void store_block_bf16(uint16_t* c, const Shape& s, int64_t bidx, int i0,
                                             int rows, int j0, int jn, int lane, const uint16_t* lh) {
    const int col = (lane & 7) * 8;
    const int rq = lane >> 3;
    const int64_t off0 = bidx * s.c_batch + static_cast<int64_t>(i0 + rq) * s.n + j0 + col;
    const int64_t step = 8 * static_cast<int64_t>(s.n);
    const bool col_ok = col < jn;
    const bool whole = VEC && col + 7 < jn;
#pragma unroll
    for (int r0 = 0; r0 < kTileM; r0 += 8) {
        const int r = r0 + rq;
        if (r < rows && col_ok) {
            const u16x8 v = *reinterpret_cast<const u16x8*>(lh + r * kLdh + col);
            uint16_t* cp = c + off0 + (r0 / 8) * step;
            if (whole) {
                __builtin_nontemporal_store(__builtin_bit_cast(u32x4, v), reinterpret_cast<u32x4*>(cp));
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    if (col + e < jn) cp[e] = v[e];
            }
        }
    }
}

// Output rows [i0, i0 + rows) (rows <= 32) of batch b, as a sequence of steps (column block,
// reduction slice); step t + 1's loads are issued before step t's arithmetic.  AREG (the
// whole reduction in one step, k <= 64): A's operands are read from LDS once, at the first
// step, and kept in registers for every column block, so later steps move only B.
template <int LAYOUT, bool BF16OUT, bool VEC, bool AREG>
__device__ __forceinline__ void rows32(const uint16_t* a, const uint16_t* b, void* c,
                                       const Shape& s, int64_t bidx, int i0, int rows, int lane,
                                       uint16_t* lds) {
    const int li = lane & 31;
    const int h = lane >> 5;
    uint16_t* const la = lds;
    uint16_t* const lb = lds + kTileM * kLdk;
    float* const lc = reinterpret_cast<float*>(lds);
    const uint16_t* a_blk = a + bidx * s.a_batch + static_cast<int64_t>(i0) * s.k;
    const uint16_t* b_blk = b + bidx * s.b_batch;
    const int nk = s.k > 0 ? (s.k + kChunkK - 1) / kChunkK : 1;  // k == 0: one step of zeros
    const int nj = (s.n + kBlockN - 1) / kBlockN;
    const int nsteps = nk * nj;
    f32x16 acc[kBlockTiles];
    // kDepth steps of operands in flight: step st + kDepth is loaded into the registers step
    // st has just written to LDS (two for the 16-byte form; the element-wise form's registers
    // allow one)
    constexpr int kDepth = VEC ? 2 : 1;
    Pieces p[kDepth];
    u16x8 a_reg[AREG ? kChunkK / kTileK : 1];
    if constexpr (AREG) {  // A once, through LDS into its MFMA layout
        u16x8 pa[kAPieces];
        load_a<VEC>(a_blk, s, rows, 0, lane, pa);
        write_a<VEC>(pa, s, rows, 0, lane, la);
        wave_lds_sync();
#pragma unroll
        for (int q = 0; q < kChunkK / kTileK; ++q)
            a_reg[q] = *reinterpret_cast<const u16x8*>(la + li * kLdk + q * kTileK + 8 * h);
        wave_lds_sync();
    }
    auto load = [&](int st, Pieces& pp) {
        const int js = st / nk, ks = st - js * nk;
        load_step<LAYOUT, VEC, !AREG>(a_blk, b_blk, s, rows, js * kBlockN, ks * kChunkK, lane, pp);
    };
#pragma unroll
    for (int d = 0; d < kDepth; ++d) {
        if (d < nsteps) load(d, p[d]);
    }
    for (int st0 = 0; st0 < nsteps; st0 += kDepth) {
#pragma unroll
    for (int d = 0; d < kDepth; ++d) {
        const int st = st0 + d;
        if (st >= nsteps) break;
        const int jb = st / nk, kb = st - jb * nk;
        const int j0 = jb * kBlockN;
        if (kb == 0) {
#pragma unroll
            for (int t = 0; t < kBlockTiles; ++t) acc[t] = f32x16{};
        }
        write_step<LAYOUT, VEC, !AREG>(p[d], s, rows, j0, kb * kChunkK, lane, la, lb);
        wave_lds_sync();
        if (st + kDepth < nsteps) load(st + kDepth, p[d]);
        const int jn = s.n - j0 < kBlockN ? s.n - j0 : kBlockN;
#pragma unroll
        for (int kk = 0; kk < kChunkK; kk += kTileK) {
            const bf16x8 av = __builtin_bit_cast(
                bf16x8, AREG ? a_reg[AREG ? kk / kTileK : 0]
                             : *reinterpret_cast<const u16x8*>(la + li * kLdk + kk + 8 * h));
#pragma unroll
            for (int t = 0; t < kBlockTiles; ++t) {  // a tile past n multiplies zeros
                bf16x8 bv;
                if constexpr (LAYOUT == kNT)
                    bv = __builtin_bit_cast(
                        bf16x8, *reinterpret_cast<const u16x8*>(lb + (t * kTileN + li) * kLdk + kk + 8 * h));
                else
                    bv = nn_row_operand(lb, t, kk, lane);
                acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bv, av, acc[t], 0, 0, 0);
            }
        }
        wave_lds_sync();  // operands consumed
        if (kb + 1 < nk) continue;
        // column block done: tile t, lane (li, h) holds output row li, columns
        // j0 + 32 t + 8 g + 4 h + 0..3
        if constexpr (BF16OUT) {  // rounded to bf16 (nearest even) on the way into LDS
            uint16_t* const lh = lds;
#pragma unroll
            for (int t = 0; t < kBlockTiles; ++t) {
#pragma unroll
                for (int g = 0; g < 4; ++g)
                    *reinterpret_cast<u32x2*>(lh + li * kLdh + t * kTileN + 8 * g + 4 * h) =
                        u32x2{pack_bf16(s.alpha * acc[t][4 * g], s.alpha * acc[t][4 * g + 1]),
                              pack_bf16(s.alpha * acc[t][4 * g + 2], s.alpha * acc[t][4 * g + 3])};
            }
            wave_lds_sync();
            store_block_bf16<VEC>(static_cast<uint16_t*>(c), s, bidx, i0, rows, j0, jn, lane, lh);
        } else {
#pragma unroll
            for (int t = 0; t < kBlockTiles; ++t) {
#pragma unroll
                for (int g = 0; g < 4; ++g)
                    *reinterpret_cast<f32x4*>(lc + li * kLdc + t * kTileN + 8 * g + 4 * h) =
                        f32x4{s.alpha * acc[t][4 * g], s.alpha * acc[t][4 * g + 1],
                              s.alpha * acc[t][4 * g + 2], s.alpha * acc[t][4 * g + 3]};
            }
            wave_lds_sync();
            store_block_f32<VEC>(static_cast<float*>(c), s, bidx, i0, rows, j0, jn, lane, lc);
        }
        wave_lds_sync();  // the next step rewrites the region
    }
    }
}

// Worker loop: worker v (a workgroup, or one wave when per_wave) runs its items; an item's
// rows are taken 32 at a time (split where a batch ends), the workgroup's waves splitting
// them when they share the item.
// Kernel modes (one compiled instance each): NT and NN, both with LDS-staged operands.
enum { kModeNt = 0, kModeNn = 1 };
constexpr int mode_lds_bytes(int) { return kLdsBytes; }
constexpr int mode_waves_per_simd(int) { return 2; }

template <int MODE, bool BF16OUT, bool VEC>
__device__ __forceinline__ void gemm_worker(const uint16_t* a, const uint16_t* b, void* c,
                                            const Shape& s, const int32_t* __restrict__ worker_ptr,
                                            const bsm_item* __restrict__ items, int per_wave,
                                            bsm_trace_rec* __restrict__ trace, uint16_t* lds_base) {
    const int w = blockIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
    const int nwaves = static_cast<int>(blockDim.x) >> 6;
    const int lane = static_cast<int>(threadIdx.x) & 63;
    const uint64_t t0 = trace ? __builtin_amdgcn_s_memrealtime() : 0;
    const int worker = per_wave ? w * nwaves + wave : w;
    const int my_wave = per_wave ? 0 : wave;
    const int my_nwaves = per_wave ? 1 : nwaves;
    uint16_t* const lds = lds_base + wave * (mode_lds_bytes(MODE) / 2);
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
                    if (VEC && s.k <= kChunkK && s.n > kBlockN)  // (registers: 16-byte form only)
                        rows32<MODE == kModeNn ? kNN : kNT, BF16OUT, VEC, true>(a, b, c, s, bidx, i, seg, lane, lds);
                    else
                        rows32<MODE == kModeNn ? kNN : kNT, BF16OUT, VEC, false>(a, b, c, s, bidx, i, seg, lane, lds);
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

extern __shared__ uint16_t bsm_gemm_lds[];  // kLdsBytes per wave

// 256-thread workgroups; each mode's instance is compiled for its waves per SIMD (registers:
// 512 / waves) and takes mode_lds_bytes() of LDS per wave.
constexpr int kGemmThreads = 256;

template <int MODE, bool BF16OUT, bool VEC>
__global__ void __launch_bounds__(kGemmThreads, mode_waves_per_simd(MODE))
bsm_gemm_kernel(const uint16_t* a, const uint16_t* b, void* c, Shape s,
                const int32_t* __restrict__ worker_ptr, const bsm_item* __restrict__ items,
                int per_wave, bsm_trace_rec* __restrict__ trace) {
    gemm_worker<MODE, BF16OUT, VEC>(a, b, c, s, worker_ptr, items, per_wave, trace, bsm_gemm_lds);
}

}  // namespace bsm_mm
