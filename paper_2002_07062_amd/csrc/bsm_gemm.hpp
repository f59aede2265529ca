// Device code of the batched matrix products around the softmax (Section 6's two batch
// matrix multiplications: scores (512 x 64) x (64 x 512) and context (512 x 512) x (512 x 64),
// batch 384), driven by the same host-built work tables as the softmax: the output C_b of
// every batch index is a slice of m rows by n columns, and an item is a run of its rows.
//
//   layout NT:  C_b = alpha A_b B_b^T   (A_b: m x k, B_b: n x k; e.g. Q K^T)
//   layout NN:  C_b = alpha A_b B_b     (A_b: m x k, B_b: k x n; e.g. P V)
//
//   NT + softmax: C_b = row softmax of alpha A_b B_b^T  (the score product with Section 2's
//                 softmax of each score row in the same kernel; S is never stored)
//
// bf16 operands, fp32 accumulation on the matrix cores (v_mfma_f32_32x32x16_bf16), fp32 or
// bf16 (round to nearest even) output.  A workgroup of four waves takes up to 128 rows of one
// batch index at a time, 32 per wave, and walks the output in blocks of 64 columns (two
// 32 x 32 MFMA tiles per wave) and the reduction in slices of 64.  Each wave computes the
// transposed tile D = B_sub A_sub^T so that a lane ends with four consecutive output columns.
// Operands are staged in LDS from 16-byte loads, two steps ahead: a wave's own A rows in its
// own region, the B block shared by the four waves (each loads a quarter of it; two buffers,
// one barrier per step); NN's B is stored as it is and read back transposed.  The output
// block goes through the wave's LDS too and is stored as whole rows.  At these shapes the
// work is bound by HBM (the 512 x 512 output, or input), not by the matrix cores.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

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
constexpr int kWaves = 4;    // waves per workgroup
constexpr int kTileM = 32;   // output rows per wave
constexpr int kTileN = 32;   // output columns per MFMA tile
constexpr int kTileK = 16;   // reduction depth per MFMA

struct Shape {
    int m, n, k;
    int64_t a_batch, b_batch, c_batch;  // elements between consecutive batch indices
    float alpha;
};

// One step of a workgroup: the output column block [j0, j0 + 64) and the reduction slice
// [k0, k0 + 64).  LDS (bf16 elements unless noted): per wave, A block [32][kLdk], reused after
// a column block's last step for the output block, [32][kLdc] fp32 or [32][kLdh] bf16; shared,
// two B buffers of [64][kLdk] (NT: B's rows) or [64][kLdv] (NN: B's rows k0 .. k0+63 as they
// are).  Rows are padded so that 16-byte accesses of consecutive rows spread over the banks.
constexpr int kChunkK = 64;                 // reduction indices per step
constexpr int kLdk = kChunkK + 8;           // padded LDS row, elements
constexpr int kBlockN = 64;                 // output columns per block (two tiles)
constexpr int kBlockTiles = kBlockN / kTileN;
constexpr int kLdc = kBlockN + 4;           // padded LDS row of the staged output, floats
constexpr int kLdh = kBlockN + 8;           // ... staged as bf16, elements
constexpr int kLdv = kBlockN + 8;           // padded LDS row of NN's B (rows = reduction index)
static_assert(kChunkK * kLdv <= kBlockN * kLdk, "NN's B fits the B buffer");
constexpr int kBBufElems = kBlockN * kLdk;  // one shared B buffer
constexpr int kDepth = 2;                   // steps of operands in flight = shared B buffers
constexpr int wave_lds_bytes(bool bf16_out) {
    return (bf16_out ? kTileM * kLdh * 2 : kTileM * kLdc * 4) > kTileM * kLdk * 2
               ? (bf16_out ? kTileM * kLdh * 2 : kTileM * kLdc * 4) : kTileM * kLdk * 2;
}
constexpr int wg_lds_bytes(bool bf16_out) { return kWaves * wave_lds_bytes(bf16_out) + kDepth * kBBufElems * 2; }
constexpr int kAPieces = kTileM * kChunkK / 8 / 64;            // 16-byte pieces of A per lane per step
constexpr int kBPieces = kBlockN * kChunkK / 8 / 64 / kWaves;  // ... of B per lane (a quarter)

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
// (cache-resident) loads where the data is read again (B by every row round of its batch, A
// by every column block), nontemporal (STREAM) where it is read once.
template <bool VEC, bool STREAM = false>
__device__ __forceinline__ u16x8 load8(const uint16_t* row, int c, int len) {
    if constexpr (VEC) {
        const u16x8* p = reinterpret_cast<const u16x8*>(row + (c < len ? c : len - 8));
        if constexpr (STREAM) return __builtin_nontemporal_load(p);
        return *p;
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
template <bool WITH_A>
struct Pieces {
    u16x8 a[WITH_A ? kAPieces : 1];
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
                                       int lane, bool stream, u16x8 (&pa)[kAPieces]) {
#pragma unroll
    for (int q = 0; q < kAPieces; ++q) {
        const int r = piece_row(lane, q);
        const uint16_t* row = a_blk + static_cast<int64_t>(r < rows ? r : (rows > 0 ? rows - 1 : 0)) * s.k;
        const int c = k0 + piece_col(lane, q);
        pa[q] = stream ? load8<VEC, true>(row, c, s.k) : load8<VEC, false>(row, c, s.k);
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

// The wave's quarter of the B block of step (j0, k0): pieces q = kBPieces * wave + 0, 1, of
// the block's 64 x 64 as 64 lanes x 8 pieces (B's rows for NT, B's rows k0.. for NN).
template <int LAYOUT, bool VEC, bool WITH_A>
__device__ __forceinline__ void load_step(const uint16_t* a_blk, const uint16_t* b_blk,
                                          const Shape& s, int rows, int j0, int k0, int wave,
                                          int lane, bool stream_a, Pieces<WITH_A>& p) {
    if constexpr (WITH_A) load_a<VEC>(a_blk, s, rows, k0, lane, stream_a, p.a);
#pragma unroll
    for (int q = 0; q < kBPieces; ++q) {
        const int qg = kBPieces * wave + q;
        if constexpr (LAYOUT == kNT) {
            const int j = j0 + piece_row(lane, qg);
            p.b[q] = load8<VEC>(b_blk + static_cast<int64_t>(j < s.n ? j : s.n - 1) * s.k,
                                k0 + piece_col(lane, qg), s.k);
        } else {
            const int kr = k0 + piece_nn_row(lane, qg);
            p.b[q] = load8<VEC>(b_blk + static_cast<int64_t>(kr < s.k ? kr : s.k - 1) * s.n,
                                j0 + piece_nn_col(lane, qg), s.n);
        }
    }
}

template <int LAYOUT, bool VEC, bool WITH_A>
__device__ __forceinline__ void write_step(const Pieces<WITH_A>& p, const Shape& s, int rows,
                                           int j0, int k0, int wave, int lane, uint16_t* la,
                                           uint16_t* lb) {
    if constexpr (WITH_A) write_a<VEC>(p.a, s, rows, k0, lane, la);
#pragma unroll
    for (int q = 0; q < kBPieces; ++q) {
        const int qg = kBPieces * wave + q;
        if constexpr (LAYOUT == kNT) {
            const int r = piece_row(lane, qg), c = piece_col(lane, qg);
            *reinterpret_cast<u16x8*>(lb + r * kLdk + c) = keep8<VEC>(p.b[q], k0 + c, s.k, j0 + r < s.n);
        } else {
            const int kr = piece_nn_row(lane, qg), c = piece_nn_col(lane, qg);
            *reinterpret_cast<u16x8*>(lb + kr * kLdv + c) = keep8<VEC>(p.b[q], j0 + c, s.n, k0 + kr < s.k);
        }
    }
}

// Stores a staged output block (rows [i0, i0 + rows), columns [j0, j0 + jn)) as whole rows:
// 16 lanes x 4 fp32 columns, four rows per instruction.
template <bool VEC, bool TEMPORAL>
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
                if constexpr (TEMPORAL)
                    *reinterpret_cast<f32x4*>(cp) = v;
                else
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
template <bool VEC, bool TEMPORAL>
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
                if constexpr (TEMPORAL)
                    *reinterpret_cast<u32x4*>(cp) = __builtin_bit_cast(u32x4, v);
                else
                    __builtin_nontemporal_store(__builtin_bit_cast(u32x4, v), reinterpret_cast<u32x4*>(cp));
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    if (col + e < jn) cp[e] = v[e];
            }
        }
    }
}

// A workgroup's round: output rows [i0, i0 + rows) of batch bidx for this wave (rows <= 32;
// 0 for a wave past the round's end, which still loads its quarter of B and meets every
// barrier), as a sequence of steps (column block, reduction slice) that all four waves take
// together; step t + kDepth's loads are issued before step t's arithmetic.  AREG (the whole
// reduction in one step, k <= 64): A's operands are read from LDS once and kept in registers
// for every column block, so later steps move only B.
// Wave priority 0..3 (s_setprio takes an immediate).  The three workgroups on a CU get the
// same rows, but the SQ favours older waves, so without this the first one dispatched finishes
// far ahead of the last (31 vs 47 us on the context product) and the CU ends on one
// workgroup's waves; each workgroup therefore lowers its priority as its own share gets done,
// and the ones behind catch up.
__device__ __forceinline__ void set_prio(int p) {
    if (p >= 3) __builtin_amdgcn_s_setprio(3);
    else if (p == 2) __builtin_amdgcn_s_setprio(2);
    else if (p == 1) __builtin_amdgcn_s_setprio(1);
    else __builtin_amdgcn_s_setprio(0);
}

constexpr float kLog2eF = 1.44269504088896340736f;
constexpr float kNegInfF = -__builtin_huge_valf();

// The value of lane l and of lane l ^ 32 (the other half of an output row's 32x32 tile
// lanes) combined by op (commutative: both lanes end with identical bits).  The partner's value
// comes through ds_bpermute: with v_permlane32_swap on two copies of one value, the compiler
// used one of the two results twice.
template <class F>
__device__ __forceinline__ float half_pair(float v, int lane, F op) {
    const float o = __builtin_bit_cast(
        float, __builtin_amdgcn_ds_bpermute((lane ^ 32) << 2, __builtin_bit_cast(int, v)));
    return op(v, o);
}

// SOFTMAX (NT only): each row's column blocks are walked twice.  The first pass keeps the
// row's running maximum M of the logits (in base-2 units, y = alpha s log2 e) and the sum of
// 2^(y - M) over the columns seen so far, rescaled whenever M rises (each lane sums its own
// columns; the two lanes of a row exchange their maxima per block and add their sums at the
// end).  The second pass recomputes the products and writes 2^(y - M) / sum.  Recomputing costs
// matrix-core time, which these products have to spare; storing S would cost its bytes twice.
template <int LAYOUT, bool BF16OUT, bool VEC, bool AREG, bool TEMPORAL, bool SOFTMAX = false>
__device__ __forceinline__ void round_rows(const uint16_t* a, const uint16_t* b, void* c,
                                           const Shape& s, int64_t bidx, int i0, int rows,
                                           int wave, int lane, uint16_t* lw, uint16_t* lbs,
                                           int done_rows, int round_rows_n, int total_rows) {
    const int li = lane & 31;
    const int h = lane >> 5;
    uint16_t* const la = lw;
    const uint16_t* a_blk = rows > 0 ? a + bidx * s.a_batch + static_cast<int64_t>(i0) * s.k : a;
    const uint16_t* b_blk = b + bidx * s.b_batch;
    const int nk = (s.k + kChunkK - 1) / kChunkK;  // k > 0 here
    const int nj = (s.n + kBlockN - 1) / kBlockN;
    const int nsteps = nk * nj;
    const int nall = (SOFTMAX ? 2 : 1) * nsteps;  // both passes' steps, in one stream
    // Accumulators are zero at every column block's start: set here and again after each
    // block's output (AREG, one step per block: the block's first MFMA takes a zero addend
    // instead), not selected at every step.
    f32x16 acc[kBlockTiles];
#pragma unroll
    for (int t = 0; t < kBlockTiles; ++t) acc[t] = f32x16{};
    Pieces<!AREG> p[kDepth];
    u16x8 a_reg[AREG ? kChunkK / kTileK : 1];
    if constexpr (AREG) {  // A once, through the wave's LDS into its MFMA layout
        u16x8 pa[kAPieces];
        load_a<VEC>(a_blk, s, rows, 0, lane, !TEMPORAL, pa);  // read once
        write_a<VEC>(pa, s, rows, 0, lane, la);
        wave_lds_sync();
#pragma unroll
        for (int q = 0; q < kChunkK / kTileK; ++q)
            a_reg[q] = *reinterpret_cast<const u16x8*>(la + li * kLdk + q * kTileK + 8 * h);
        wave_lds_sync();
    }
    // The steps' (column block, reduction slice) pairs are counted up as the steps go, not
    // divided out of the step index: on this path every scalar instruction counts, twelve
    // waves per CU share the scalar unit.  The load stream runs kDepth steps ahead and stays
    // on the last step once it gets there (its loads are then issued again, unused).
    int ld_st = 0, ld_j = 0, ld_k = 0;
    auto load = [&](Pieces<!AREG>& pp) {
        load_step<LAYOUT, VEC, !AREG>(a_blk, b_blk, s, rows, ld_j * kBlockN, ld_k * kChunkK, wave, lane,
                                      !TEMPORAL && nj == 1, pp);  // A read once when one column block
        if (ld_st + 1 < nall) {
            ++ld_st;
            if (++ld_k == nk) {
                ld_k = 0;
                if (++ld_j == nj) ld_j = 0;  // the second pass starts again at block 0
            }
        }
    };
#pragma unroll
    for (int d = 0; d < kDepth; ++d) load(p[d]);
    static_assert(kDepth == 2, "the step loop below is written for two buffers");
    // Wave priority 3 .. 0 by the workgroup's own progress: step st of this round has done
    // done_rows * nsteps + round_rows_n * st of total_rows * nsteps row-steps, and the
    // priority is 3 - floor(4 done / total) (at least 0).  The steps where the quotient
    // reaches 1, 2 and 3 are worked out once per round (measured: -2.5% time on the context
    // product; the one-step scores product gains nothing and skips it).
    int prio_step[3] = {0, 0, 0};
    if constexpr (!AREG) {
        const int64_t tot = static_cast<int64_t>(total_rows > 0 ? total_rows : 1) * nall;
        const int64_t done4 = 4 * static_cast<int64_t>(done_rows) * nall;
        const int64_t per4 = 4 * static_cast<int64_t>(round_rows_n > 0 ? round_rows_n : 1);
#pragma unroll
        for (int q = 0; q < 3; ++q) {
            const int64_t need = (q + 1) * tot - done4;  // 4 * row-steps still short of q + 1
            const int64_t t = need <= 0 ? 0 : (need + per4 - 1) / per4;
            prio_step[q] = t < nall ? static_cast<int>(t) : nall;
        }
    }
    int cur_j = 0, cur_k = 0;
    float sm_max = kNegInfF, sm_sum = 0.0f, sm_inv = 0.0f;  // SOFTMAX: this lane's row
    // One step: st's operands (in pp, loaded kDepth steps ago) go to LDS buffer lb, then
    // step st + kDepth's loads are issued into pp, then st's arithmetic and, at a column
    // block's end, its output.
    // PASS (a compile-time tag): 0 without SOFTMAX, else 1 (row statistics) or 2 (output), so
    // that each pass's step is compiled on its own.
    auto step = [&](auto pass, int st, Pieces<!AREG>& pp, uint16_t* lb) {
        constexpr int PASS = decltype(pass)::value;
        if constexpr (!AREG)
            set_prio(3 - (st >= prio_step[0]) - (st >= prio_step[1]) - (st >= prio_step[2]));
        const int jb = cur_j, kb = cur_k;
        if (++cur_k == nk) {
            cur_k = 0;
            if (++cur_j == nj) cur_j = 0;
        }
        const int j0 = jb * kBlockN;
        // lb (buffer st % 2) was last read at step st - 2; every wave finished that step
        // before the barrier of step st - 1, so one barrier per step orders both uses.
        write_step<LAYOUT, VEC, !AREG>(pp, s, rows, j0, kb * kChunkK, wave, lane, la, lb);
        __syncthreads();
        // issued on every step (past the last step: the last step's operands again, cache
        // hits, unused), so that every path has the same loads in flight
        load(pp);
        if (rows > 0) {  // wave-uniform
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
                    acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        bv, av, (AREG && kk == 0) ? f32x16{} : acc[t], 0, 0, 0);
                }
            }
        }
        wave_lds_sync();  // the wave's A consumed
        if (kb + 1 < nk || rows == 0) return;
        // column block done: tile t, lane (li, h) holds output row li, columns
        // j0 + 32 t + 8 g + 4 h + 0..3
        const int jn = s.n - j0 < kBlockN ? s.n - j0 : kBlockN;
        float scale = s.alpha;
        if constexpr (SOFTMAX) {
            // Logits in base-2 units, y = acc * c with c = alpha log2 e, never formed on their
            // own: the row maximum of y is c times the maximum (c < 0: minimum) of acc, and each
            // 2^(y - M) takes one fma and one v_exp_f32.  Columns past n (a partial last block)
            // count as -inf.
            const float c2 = s.alpha * kLog2eF;
            const bool full = jn == kBlockN;  // wave-uniform: only a partial last block masks
            auto col_ok = [&](int t, int i) { return t * kTileN + 8 * (i / 4) + 4 * h + (i % 4) < jn; };
            if constexpr (PASS == 1) {  // first pass: fold this block into the row's maximum and sum
                // the block's largest y is c times its largest (c < 0: smallest) product; the four
                // loops leave acc untouched, so no branch needs copies of it
                auto extreme = [&](auto pick, float none) {
                    float e = none;
                    if (full) {
#pragma unroll
                        for (int t = 0; t < kBlockTiles; ++t)
#pragma unroll
                            for (int i = 0; i < 16; ++i) e = pick(e, acc[t][i]);
                    } else {
#pragma unroll
                        for (int t = 0; t < kBlockTiles; ++t)
#pragma unroll
                            for (int i = 0; i < 16; ++i) e = pick(e, col_ok(t, i) ? acc[t][i] : none);
                    }
                    return e;
                };
                float bm = c2 >= 0.0f
                               ? extreme([](float u, float v) { return __builtin_elementwise_maximum(u, v); }, kNegInfF)
                               : extreme([](float u, float v) { return __builtin_elementwise_minimum(u, v); }, -kNegInfF);
                bm = c2 == 0.0f ? 0.0f : c2 * bm;  // the block's largest y (alpha = 0: all y are 0)
                bm = half_pair(bm, lane, [](float u, float v) { return __builtin_elementwise_maximum(u, v); });
                const float mx = __builtin_elementwise_maximum(sm_max, bm);
                const float ms = mx == kNegInfF ? 0.0f : mx;
#pragma unroll
                for (int t = 0; t < kBlockTiles; ++t)
#pragma unroll
                    for (int i = 0; i < 16; ++i) acc[t][i] = __builtin_amdgcn_exp2f(__builtin_fmaf(acc[t][i], c2, -ms));
                if (!full) {  // columns past n add nothing
#pragma unroll
                    for (int t = 0; t < kBlockTiles; ++t)
#pragma unroll
                        for (int i = 0; i < 16; ++i)
                            if (!col_ok(t, i)) acc[t][i] = 0.0f;
                }
                // pairwise sum of the lane's 32 values: within each tile 16 -> 1, then the tiles
#pragma unroll
                for (int t = 0; t < kBlockTiles; ++t)
#pragma unroll
                    for (int w = 8; w >= 1; w /= 2)
#pragma unroll
                        for (int i = 0; i < w; ++i) acc[t][i] = acc[t][2 * i] + acc[t][2 * i + 1];
                static_assert(kBlockTiles == 2, "two tiles per block");
                const float bs = acc[0][0] + acc[1][0];
                sm_sum = sm_sum * __builtin_amdgcn_exp2f(sm_max - ms) + bs;
                sm_max = mx;
                if (jb + 1 == nj) {  // the row's last block: both lanes' sums, and 1 / sum
                    const float tot = half_pair(sm_sum, lane, [](float u, float v) { return u + v; });
                    sm_inv = tot == 0.0f ? 0.0f : __builtin_amdgcn_rcpf(tot);
                }
                if constexpr (!AREG) {
#pragma unroll
                    for (int t = 0; t < kBlockTiles; ++t) acc[t] = f32x16{};
                }
                return;
            }
            // second pass: the block's probabilities, then the ordinary output path
            const float ms = sm_max == kNegInfF ? 0.0f : sm_max;
#pragma unroll
            for (int t = 0; t < kBlockTiles; ++t)
#pragma unroll
                for (int i = 0; i < 16; ++i)
                    acc[t][i] = __builtin_amdgcn_exp2f(__builtin_fmaf(acc[t][i], c2, -ms)) * sm_inv;
            scale = 1.0f;
        }
        if constexpr (BF16OUT) {  // rounded to bf16 (nearest even) on the way into LDS
            uint16_t* const lh = lw;
#pragma unroll
            for (int t = 0; t < kBlockTiles; ++t) {
#pragma unroll
                for (int g = 0; g < 4; ++g)
                    *reinterpret_cast<u32x2*>(lh + li * kLdh + t * kTileN + 8 * g + 4 * h) =
                        u32x2{pack_bf16(scale * acc[t][4 * g], scale * acc[t][4 * g + 1]),
                              pack_bf16(scale * acc[t][4 * g + 2], scale * acc[t][4 * g + 3])};
            }
            wave_lds_sync();
            store_block_bf16<VEC, TEMPORAL>(static_cast<uint16_t*>(c), s, bidx, i0, rows, j0, jn, lane, lh);
        } else {
            float* const lc = reinterpret_cast<float*>(lw);
#pragma unroll
            for (int t = 0; t < kBlockTiles; ++t) {
#pragma unroll
                for (int g = 0; g < 4; ++g)
                    *reinterpret_cast<f32x4*>(lc + li * kLdc + t * kTileN + 8 * g + 4 * h) =
                        f32x4{scale * acc[t][4 * g], scale * acc[t][4 * g + 1],
                              scale * acc[t][4 * g + 2], scale * acc[t][4 * g + 3]};
            }
            wave_lds_sync();
            store_block_f32<VEC, TEMPORAL>(static_cast<float*>(c), s, bidx, i0, rows, j0, jn, lane, lc);
        }
        wave_lds_sync();  // the next step rewrites the region
        if constexpr (!AREG) {
#pragma unroll
            for (int t = 0; t < kBlockTiles; ++t) acc[t] = f32x16{};
        }
    };
    // Two steps per iteration and the odd one after the loop, so that every path around the
    // loop issues the same loads (a step waits for its own loads only, not for the next
    // step's, which the wait-count insertion would otherwise have to assume).
    // With SOFTMAX the second pass continues the same buffer order: it starts on buffer 1
    // when the first pass has an odd number of steps.
    using P0 = std::integral_constant<int, 0>;
    using P1 = std::integral_constant<int, 1>;
    using P2 = std::integral_constant<int, 2>;
    // Step 0 writes buffer 0, which the previous round's last step read when a round has an odd
    // number of steps (every round of a launch has the same number): then one more barrier, so
    // that no wave still reads it.
    if (nall & 1) __syncthreads();
    int st = 0;
    auto run = [&](auto pass, int end, bool odd_start) {
        if (!odd_start) {
            for (; st + 1 < end; st += 2) {
                step(pass, st, p[0], lbs);
                step(pass, st + 1, p[1], lbs + kBBufElems);
            }
            if (st < end) step(pass, st++, p[0], lbs);
        } else {
            for (; st + 1 < end; st += 2) {
                step(pass, st, p[1], lbs + kBBufElems);
                step(pass, st + 1, p[0], lbs);
            }
            if (st < end) step(pass, st++, p[1], lbs + kBBufElems);
        }
    };
    if constexpr (!SOFTMAX) {
        run(P0{}, nall, false);
    } else {
        run(P1{}, nsteps, false);
        run(P2{}, nall, (nsteps & 1) != 0);
    }
}

// An empty reduction (k == 0): the wave's output rows are zeros, or with SOFTMAX the
// softmax of a row of zero logits, 1/n (as the two passes compute it: 2^0 times 1 / n).
template <bool BF16OUT, bool SOFTMAX>
__device__ __forceinline__ void zero_rows(void* c, const Shape& s, int64_t bidx, int i0, int rows,
                                          int lane) {
    const float v = SOFTMAX ? __builtin_amdgcn_rcpf(static_cast<float>(s.n)) : 0.0f;
    for (int r = 0; r < rows; ++r) {
        const int64_t off = bidx * s.c_batch + static_cast<int64_t>(i0 + r) * s.n;
        for (int j = lane; j < s.n; j += 64) {
            if constexpr (BF16OUT)
                static_cast<uint16_t*>(c)[off + j] = static_cast<uint16_t>(pack_bf16(v, 0.0f) & 0xFFFFu);
            else
                static_cast<float*>(c)[off + j] = v;
        }
    }
}

// ----------------------------------------------------------- single-pass score softmax
// NT + softmax for k <= 128 and 64 < n <= 512 (Section 6's score shape, d = 64 over sequences of
// up to 512): each product is formed once and held in registers until its row is done.  The
// two waves of a pair share 32 output rows; wave q of the pair takes the column blocks 2s + q
// (s = 0 .. 3), so a step stages 128 rows of B (two 64-column blocks) and each wave holds at
// most four blocks, 128 values per lane.  A row's maximum and sum are combined between the two
// lanes of its row (half_pair) and the two waves of its pair (LDS), then the held values are
// turned into probabilities and stored block by block.  Two waves per SIMD (the held values
// take 128 registers); a workgroup round covers 64 rows.
constexpr int kS1Rows = 2 * kTileM;                                // rows per workgroup round
constexpr int kS1BlockN = 2 * kBlockN;                             // B rows staged per step
constexpr int kS1MaxSteps = 4;                                     // n <= 4 * 128
constexpr int kS1BBufElems = kS1BlockN * kLdk;
constexpr int kS1BPieces = kS1BlockN * kChunkK / 8 / 64 / kWaves;  // 16-byte pieces per lane
constexpr int kS1WavesPerSimd = 2;
// DEEP (64 < k <= 128): the wave's 32 A rows stay in its LDS region for the round (pitch
// kLdA) and each 128-column step takes two 64-deep chunks of B through the shared buffers.
constexpr int kLdA = 2 * kChunkK + 8;
constexpr int s1_wave_bytes(bool bf16_out, bool deep) {
    return deep && kTileM * kLdA * 2 > wave_lds_bytes(bf16_out) ? kTileM * kLdA * 2 : wave_lds_bytes(bf16_out);
}
constexpr int s1_lds_bytes(bool bf16_out, bool deep = false) {
    return kWaves * s1_wave_bytes(bf16_out, deep) + kDepth * kS1BBufElems * 2 + 2 * kWaves * kTileM * 4;
}
constexpr bool single_pass_shape(int n, int k) {
    return k > 0 && k <= 2 * kChunkK && n > kBlockN && n <= kS1MaxSteps * kS1BlockN;
}

struct S1Pieces {
    u16x8 b[kS1BPieces];
};

// The wave's quarter of B's rows [j0, j0 + 128), reduction slice [k0, k0 + 64), and its LDS
// write (rows past n and columns past k zeroed).
__device__ __forceinline__ void s1_load(const uint16_t* b_blk, const Shape& s, int j0, int k0, int wave,
                                        int lane, S1Pieces& p) {
#pragma unroll
    for (int q = 0; q < kS1BPieces; ++q) {
        const int qg = kS1BPieces * wave + q;
        const int j = j0 + piece_row(lane, qg);
        p.b[q] = load8<true>(b_blk + static_cast<int64_t>(j < s.n ? j : s.n - 1) * s.k,
                             k0 + piece_col(lane, qg), s.k);
    }
}

__device__ __forceinline__ void s1_write(const S1Pieces& p, const Shape& s, int j0, int k0, int wave,
                                         int lane, uint16_t* lb) {
#pragma unroll
    for (int q = 0; q < kS1BPieces; ++q) {
        const int qg = kS1BPieces * wave + q;
        const int r = piece_row(lane, qg), c = piece_col(lane, qg);
        *reinterpret_cast<u16x8*>(lb + r * kLdk + c) = keep8<true>(p.b[q], k0 + c, s.k, j0 + r < s.n);
    }
}

// Stages one output block (two 32 x 32 tiles, times `scale`) in the wave's LDS region and
// stores it as whole rows.
template <bool BF16OUT, bool TEMPORAL>
__device__ __forceinline__ void s1_store_block(const f32x16 (&v)[kBlockTiles], float scale, void* c,
                                               const Shape& s, int64_t bidx, int i0, int rows,
                                               int j0, int jn, int lane, uint16_t* lw) {
    const int li = lane & 31, h = lane >> 5;
    if constexpr (BF16OUT) {
#pragma unroll
        for (int t = 0; t < kBlockTiles; ++t)
#pragma unroll
            for (int g = 0; g < 4; ++g)
                *reinterpret_cast<u32x2*>(lw + li * kLdh + t * kTileN + 8 * g + 4 * h) =
                    u32x2{pack_bf16(scale * v[t][4 * g], scale * v[t][4 * g + 1]),
                          pack_bf16(scale * v[t][4 * g + 2], scale * v[t][4 * g + 3])};
        wave_lds_sync();
        store_block_bf16<true, TEMPORAL>(static_cast<uint16_t*>(c), s, bidx, i0, rows, j0, jn, lane, lw);
    } else {
        float* const lc = reinterpret_cast<float*>(lw);
#pragma unroll
        for (int t = 0; t < kBlockTiles; ++t)
#pragma unroll
            for (int g = 0; g < 4; ++g)
                *reinterpret_cast<f32x4*>(lc + li * kLdc + t * kTileN + 8 * g + 4 * h) =
                    f32x4{scale * v[t][4 * g], scale * v[t][4 * g + 1], scale * v[t][4 * g + 2],
                          scale * v[t][4 * g + 3]};
        wave_lds_sync();
        store_block_f32<true, TEMPORAL>(static_cast<float*>(c), s, bidx, i0, rows, j0, jn, lane, lc);
    }
    wave_lds_sync();  // the next block rewrites the region
}

// One round of a wave: output rows [i0, i0 + rows) of batch bidx (rows <= 32; 0 for a wave
// past the round's end, which still loads its part of B and meets every barrier).  lstat:
// [2][kWaves][32] floats, the waves' row maxima and sums for their partners.
template <bool BF16OUT, bool TEMPORAL, bool DEEP>
__device__ __forceinline__ void round_rows_s1(const uint16_t* a, const uint16_t* b, void* c,
                                              const Shape& s, int64_t bidx, int i0, int rows,
                                              int wave, int lane, uint16_t* lw, uint16_t* lbs,
                                              float* lstat) {
    const int li = lane & 31;
    const int h = lane >> 5;
    const int q = wave & 1;
    const uint16_t* a_blk = rows > 0 ? a + bidx * s.a_batch + static_cast<int64_t>(i0) * s.k : a;
    const uint16_t* b_blk = b + bidx * s.b_batch;
    const int nj = (s.n + kBlockN - 1) / kBlockN;  // 2 .. 8
    const int ns = (nj + 1) / 2;                   // steps: 1 .. 4
    // Sub-steps: chunk kc (64 deep) of step st is sub-step NK st + kc (NK = 2 with DEEP).
    constexpr int NK = DEEP ? 2 : 1;
    const int nu = NK * ns;
    auto sub_j0 = [](int u) { return (u / NK) * kS1BlockN; };
    auto sub_k0 = [](int u) { return (u % NK) * kChunkK; };
    // A's rows and B's first two sub-steps.  Both waves of a pair read the same A rows:
    // ordinary loads, so that the second finds them in cache.
    u16x8 pa[NK][kAPieces];
#pragma unroll
    for (int kc = 0; kc < NK; ++kc) load_a<true>(a_blk, s, rows, kc * kChunkK, lane, false, pa[kc]);
    S1Pieces p[kDepth];
    s1_load(b_blk, s, sub_j0(0), sub_k0(0), wave, lane, p[0]);
    s1_load(b_blk, s, sub_j0(nu > 1 ? 1 : 0), sub_k0(nu > 1 ? 1 : 0), wave, lane, p[1]);
    // A through the wave's LDS into its MFMA layout: into registers (k <= 64), or kept there
    // for the round (DEEP, row pitch kLdA)
    constexpr int LDA = DEEP ? kLdA : kLdk;
#pragma unroll
    for (int kc = 0; kc < NK; ++kc) {
#pragma unroll
        for (int qq = 0; qq < kAPieces; ++qq) {
            const int r = piece_row(lane, qq), cc = piece_col(lane, qq);
            *reinterpret_cast<u16x8*>(lw + r * LDA + kc * kChunkK + cc) =
                keep8<true>(pa[kc][qq], kc * kChunkK + cc, s.k, r < rows);
        }
    }
    wave_lds_sync();
    u16x8 a_reg[DEEP ? 1 : kChunkK / kTileK];
    if constexpr (!DEEP) {
#pragma unroll
        for (int kq = 0; kq < kChunkK / kTileK; ++kq)
            a_reg[kq] = *reinterpret_cast<const u16x8*>(lw + li * kLdk + kq * kTileK + 8 * h);
        wave_lds_sync();
    }
    f32x16 held[kS1MaxSteps][kBlockTiles];
#pragma unroll
    for (int st = 0; st < kS1MaxSteps; ++st) {
        if (st >= ns) break;  // wave-uniform
#pragma unroll
        for (int kc = 0; kc < NK; ++kc) {
            const int u = NK * st + kc;
            uint16_t* const lb = lbs + (u & 1) * kS1BBufElems;
            // Buffer u % 2 was last read at sub-step u - 2, which every wave finished before the
            // barrier of sub-step u - 1; the previous round's last reads came before its
            // row-statistics barriers.
            s1_write(p[u & 1], s, sub_j0(u), sub_k0(u), wave, lane, lb);
            __syncthreads();
            // sub-step u + 2's operands (none past the last)
            if (u + 2 < nu) s1_load(b_blk, s, sub_j0(u + 2), sub_k0(u + 2), wave, lane, p[u & 1]);
#pragma unroll
            for (int kk = 0; kk < kChunkK; kk += kTileK) {
                bf16x8 av;
                if constexpr (DEEP)
                    av = __builtin_bit_cast(
                        bf16x8, *reinterpret_cast<const u16x8*>(lw + li * kLdA + kc * kChunkK + kk + 8 * h));
                else
                    av = __builtin_bit_cast(bf16x8, a_reg[DEEP ? 0 : kk / kTileK]);
#pragma unroll
                for (int t = 0; t < kBlockTiles; ++t) {  // a tile past n multiplies zeros
                    const bf16x8 bv = __builtin_bit_cast(
                        bf16x8, *reinterpret_cast<const u16x8*>(lb + (q * kBlockN + t * kTileN + li) * kLdk + kk + 8 * h));
                    held[st][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        bv, av, (kc == 0 && kk == 0) ? f32x16{} : held[st][t], 0, 0, 0);
                }
            }
        }
    }
    if constexpr (DEEP) wave_lds_sync();  // the wave's A consumed before its output staging
    // Tile t of step st, lane (li, h): row li, columns 64 (2 st + q) + 32 t + 8 g + 4 h + 0..3
    // (value 4 g + e).  Blocks past n (st >= ns, or wave 1 of a pair past an odd block count)
    // take no part.
    auto block_cols = [&](int st) {
        const int j0 = (2 * st + q) * kBlockN;
        return st < ns && j0 < s.n ? (s.n - j0 < kBlockN ? s.n - j0 : kBlockN) : 0;
    };
    auto col_ok = [&](int jn, int t, int i) { return t * kTileN + 8 * (i / 4) + 4 * h + (i % 4) < jn; };
    // Logits in base-2 units, y = c2 * product (alpha != 0: the host sends alpha = 0 to the
    // two-pass form).  Columns past n inside a partial block get a product whose y is -inf,
    // once, so that the maximum, the exponentials and the sums below take every held value as
    // it is.
    const float c2 = s.alpha * kLog2eF;
    const float none = c2 > 0.0f ? kNegInfF : -kNegInfF;
#pragma unroll
    for (int st = 0; st < kS1MaxSteps; ++st) {
        const int jn = block_cols(st);
        if (jn > 0 && jn < kBlockN) {
#pragma unroll
            for (int t = 0; t < kBlockTiles; ++t)
#pragma unroll
                for (int i = 0; i < 16; ++i) held[st][t][i] = col_ok(jn, t, i) ? held[st][t][i] : none;
        }
    }
    // the row's largest y: c2 times its largest (c2 < 0: smallest) product, pairwise (16 -> 1
    // per tile, then the tiles) rather than one chain of 128
    auto extreme = [&](auto pick, float none) {
        float part[kS1MaxSteps * kBlockTiles];
#pragma unroll
        for (int st = 0; st < kS1MaxSteps; ++st) {
#pragma unroll
            for (int t = 0; t < kBlockTiles; ++t) {
                part[st * kBlockTiles + t] = none;
                if (block_cols(st) > 0) {
                    float f[16];
#pragma unroll
                    for (int i = 0; i < 16; ++i) f[i] = held[st][t][i];
#pragma unroll
                    for (int w = 8; w >= 1; w /= 2)
#pragma unroll
                        for (int i = 0; i < w; ++i) f[i] = pick(f[2 * i], f[2 * i + 1]);
                    part[st * kBlockTiles + t] = f[0];
                }
            }
        }
#pragma unroll
        for (int w = kS1MaxSteps * kBlockTiles / 2; w >= 1; w /= 2)
#pragma unroll
            for (int i = 0; i < w; ++i) part[i] = pick(part[2 * i], part[2 * i + 1]);
        return part[0];
    };
    float bm = c2 > 0.0f
                   ? extreme([](float u, float v) { return __builtin_elementwise_maximum(u, v); }, kNegInfF)
                   : extreme([](float u, float v) { return __builtin_elementwise_minimum(u, v); }, -kNegInfF);
    bm = c2 * bm;
    bm = half_pair(bm, lane, [](float u, float v) { return __builtin_elementwise_maximum(u, v); });
    float* const lmax = lstat;
    float* const lsum = lstat + kWaves * kTileM;
    if (h == 0) lmax[wave * kTileM + li] = bm;
    __syncthreads();
    const float mx = __builtin_elementwise_maximum(bm, lmax[(wave ^ 1) * kTileM + li]);
    const float ms = mx == kNegInfF ? 0.0f : mx;
    // 2^(y - M) in place (0 past n), and the lane's sum: 16 -> 1 per tile, then the tiles
    float part[kS1MaxSteps * kBlockTiles];
#pragma unroll
    for (int st = 0; st < kS1MaxSteps; ++st) {
#pragma unroll
        for (int t = 0; t < kBlockTiles; ++t) {
            part[st * kBlockTiles + t] = 0.0f;
            if (block_cols(st) > 0) {
#pragma unroll
                for (int i = 0; i < 16; ++i)
                    held[st][t][i] = __builtin_amdgcn_exp2f(__builtin_fmaf(held[st][t][i], c2, -ms));
                float f[16];
#pragma unroll
                for (int i = 0; i < 16; ++i) f[i] = held[st][t][i];
#pragma unroll
                for (int w = 8; w >= 1; w /= 2)
#pragma unroll
                    for (int i = 0; i < w; ++i) f[i] = f[2 * i] + f[2 * i + 1];
                part[st * kBlockTiles + t] = f[0];
            }
        }
    }
#pragma unroll
    for (int w = kS1MaxSteps * kBlockTiles / 2; w >= 1; w /= 2)
#pragma unroll
        for (int i = 0; i < w; ++i) part[i] = part[2 * i] + part[2 * i + 1];
    const float bs = half_pair(part[0], lane, [](float u, float v) { return u + v; });
    if (h == 0) lsum[wave * kTileM + li] = bs;
    __syncthreads();
    const float tot = bs + lsum[(wave ^ 1) * kTileM + li];
    const float inv = tot == 0.0f ? 0.0f : __builtin_amdgcn_rcpf(tot);
    if (rows == 0) return;  // wave-uniform; every barrier of the round is behind
#pragma unroll
    for (int st = 0; st < kS1MaxSteps; ++st) {
        const int jn = block_cols(st);
        if (jn > 0)
            s1_store_block<BF16OUT, TEMPORAL>(held[st], inv, c, s, bidx, i0, rows, (2 * st + q) * kBlockN,
                                              jn, lane, lw);
    }
}

// Kernel modes (one compiled instance each): NT, NN, NT with the row softmax in two passes,
// and in one pass (single_pass_shape).
enum { kModeNt = 0, kModeNn = 1, kModeNtSoftmax = 2, kModeNtSoftmax1 = 3 };
constexpr int kWavesPerSimd = 3;

// Worker loop: workgroup w runs its items; an item's rows are taken up to 128 at a time (cut
// where a batch ends), 32 per wave (single-pass softmax: 64 at a time, 32 per wave pair).  Every bound of these loops is the same for the four
// waves, so they meet the same barriers.
template <int MODE, bool BF16OUT, bool VEC, bool TEMPORAL, bool AREG>
__device__ __forceinline__ void gemm_worker(const uint16_t* a, const uint16_t* b, void* c,
                                            const Shape& s, const int32_t* __restrict__ worker_ptr,
                                            const bsm_item* __restrict__ items,
                                            bsm_trace_rec* __restrict__ trace, uint16_t* lds_base) {
    constexpr int kLayout = MODE == kModeNn ? kNN : kNT;
    constexpr bool kSoftmax = MODE == kModeNtSoftmax;
    constexpr bool kS1 = MODE == kModeNtSoftmax1;
    static_assert(!kS1 || VEC, "the single-pass form is a 16-byte instance");
    // The single-pass instances take their last template flag as the deep form (64 < k <= 128,
    // A kept in LDS), not as A in registers, which their k <= 64 form always does.
    constexpr bool kDeep = kS1 && AREG;
    constexpr int kRoundRows = kS1 ? kS1Rows : kWaves * kTileM;
    const int w = blockIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
    const int lane = static_cast<int>(threadIdx.x) & 63;
    const uint64_t t0 = trace ? __builtin_amdgcn_s_memrealtime() : 0;
    constexpr int kWaveBytes = kS1 ? s1_wave_bytes(BF16OUT, kDeep) : wave_lds_bytes(BF16OUT);
    uint16_t* const lw = lds_base + wave * (kWaveBytes / 2);
    uint16_t* const lbs = lds_base + kWaves * (kWaveBytes / 2);
    float* const lstat = reinterpret_cast<float*>(lbs + kDepth * kS1BBufElems);  // kS1 only
    const int row0 = kS1 ? (wave >> 1) * kTileM : wave * kTileM;  // the wave's first row of a round
    uint32_t done = 0;
    const int i_begin = worker_ptr[w];
    const int i_end = worker_ptr[w + 1];
    int total_rows = 0, wg_done = 0;
    for (int it = i_begin; it < i_end; ++it) total_rows += items[it].nrows * items[it].reps;
    for (int it = i_begin; it < i_end; ++it) {
        const int64_t e0 = items[it].elem_offset;
        const int nrows = items[it].nrows;
        const int reps = items[it].reps;
        const int64_t stride = static_cast<int64_t>(items[it].rep_stride) * s.n;
        for (int r = 0; r < reps; ++r) {
            // Output rows are numbered batch after batch (row G = b m + i); a run may cross
            // from one batch into the next.
            int64_t g = (e0 + r * stride) / s.n;
            int left = nrows;
            while (left > 0) {
                const int64_t bidx = g / s.m;
                const int i = static_cast<int>(g - bidx * s.m);
                int seg = s.m - i < left ? s.m - i : left;
                if (seg > kRoundRows) seg = kRoundRows;
                int mine = seg - row0;
                mine = mine < 0 ? 0 : (mine > kTileM ? kTileM : mine);
                if constexpr (kS1) {  // k > 0 and alpha != 0 (the host picks this form only then)
                    round_rows_s1<BF16OUT, TEMPORAL, kDeep>(a, b, c, s, bidx, i + row0, mine, wave, lane, lw,
                                                     lbs, lstat);
                } else {
                    if (s.k == 0)
                        zero_rows<BF16OUT, kSoftmax>(c, s, bidx, i + row0, mine, lane);
                    else
                        round_rows<kLayout, BF16OUT, VEC, AREG, TEMPORAL, kSoftmax>(
                            a, b, c, s, bidx, i + row0, mine, wave, lane, lw, lbs, wg_done, seg, total_rows);
                }
                wg_done += seg;
                // one-pass softmax: the two waves of a pair share rows; the first counts them
                if (!kS1 || (wave & 1) == 0) done += static_cast<uint32_t>(mine);
                g += seg;
                left -= seg;
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
        trace[static_cast<int64_t>(w) * kWaves + wave] = rec;
    }
}

extern __shared__ uint16_t bsm_gemm_lds[];  // wg_lds_bytes() per workgroup

constexpr int kGemmThreads = 64 * kWaves;

// The element-wise (unaligned / odd-size) form is compiled for two waves per SIMD: its
// registers do not fit three; so is the single-pass softmax, whose held products take 128, and
// the two-pass softmax with A staged through LDS (k > 64): capped at three waves it spilled 149
// registers and took 157 us at 192 x 512 x 512 x 128, against 83 us at two.
// TEMPORAL: ordinary stores of C and loads of A (a consumer finds C in the Infinity Cache)
// instead of nontemporal ones; a compile-time choice, so the default instance carries no
// branch for it.  AREG (A's operands held in registers, k <= 64 < n, 16-byte form only): a
// separate instance too, so that neither form's registers are allocated for the other's.
constexpr bool use_areg(bool vec, int n, int k) { return vec && k <= kChunkK && n > kBlockN; }
template <int MODE, bool BF16OUT, bool VEC, bool TEMPORAL, bool AREG>
__global__ void __launch_bounds__(kGemmThreads,
                                  (MODE == kModeNtSoftmax1 || !VEC || (MODE == kModeNtSoftmax && !AREG))
                                      ? kS1WavesPerSimd : kWavesPerSimd)
bsm_gemm_kernel(const uint16_t* a, const uint16_t* b, void* c, Shape s,
                const int32_t* __restrict__ worker_ptr, const bsm_item* __restrict__ items,
                bsm_trace_rec* __restrict__ trace) {
    static_assert(VEC || !AREG, "registers hold A in the 16-byte form only");
    gemm_worker<MODE, BF16OUT, VEC, TEMPORAL, AREG>(a, b, c, s, worker_ptr, items, trace, bsm_gemm_lds);
}

}  // namespace bsm_mm
