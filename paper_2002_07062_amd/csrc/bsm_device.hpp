// Device code of the persistent batched row-softmax kernels for gfx950 (CDNA4, wave64).
//
// One launch runs a grid of n_wg persistent workgroups.  Each worker -- a workgroup, or a
// single wave when the table is per-wave -- walks its items [worker_ptr[v], worker_ptr[v+1])
// of the host-built work table (the mapping table of the paper's Section 5: geometry is read
// per item, the instructions are the same for every patch).  A row up to the register tile is
// owned by one group of lanes of one wave (no barrier); a longer row is shared by all the
// waves of its workgroup (256 or 512 threads), which combine their partial max and sum through
// LDS.
//
// Per row (softmax over the row, the operation of the problem statement, Section 2):
//   128-bit loads (fp32, or bf16 widened to fp32; nontemporal unless the plan asks for cache-
//   resident accesses) -> lane max -> group max (DPP,
//   permlane) -> e = 2^((x - m) * log2 e) (v_exp_f32) -> lane sum (pairwise) -> group sum
//   -> y = e * (1/S) -> round-to-nearest-even to bf16 if needed -> 128-bit stores.
// Reductions combine each lane with a partner that combines the same two values in the other
// order; IEEE max and add are commutative, so every lane of a group ends with the same bits,
// and a row's result depends only on its values and length, never on the schedule.
//
// A group of G lanes (16, 32 or 64) owns one row and holds V 16-byte vectors per lane, so a
// wave covers 64/G rows at a time, with four 16-byte loads per lane in flight.  Rows longer
// than the largest register tile (512 vectors) are held in the registers of a whole workgroup
// (up to 32 values per lane in kernel class 4, 64 in classes 5 and 6, whose workgroups have 256
// and 512 threads) and read once, or, longer still, read twice with an online max/sum.  Rows whose start or length is not 16-byte aligned use
// element loads with the same lane layout, or one wave per row (staged in the wave's LDS
// region, else two passes).  This is bandwidth-bound work: no MFMA.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "bsm.h"
#include "bsm_tile.hpp"

// No multiply-add contraction anywhere in this code: the same row may run through different
// instances (a tile's U-row and one-row forms), and a fused a*b+c in one of them would round
// differently from the other, so a row's bits would depend on the schedule.
#pragma clang fp contract(off)

namespace bsm_dev {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.44269504088896340736f;
constexpr float kNegInf = -__builtin_huge_valf();

__device__ __forceinline__ float bits_f(unsigned v) { return __builtin_bit_cast(float, v); }
__device__ __forceinline__ unsigned f_bits(float v) { return __builtin_bit_cast(unsigned, v); }

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
    return __builtin_bit_cast(
        float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, true));
}

// The row max uses IEEE 754-2019 maximum (NaN in, NaN out: gfx950's v_maximum3_f32), not
// fmaxf: fmaxf's NaN-ignoring form makes the compiler canonicalize every operand first (one
// extra instruction per value and per butterfly stage).  A NaN anywhere in the row makes the
// whole row NaN either way (through the max here, through the exponentials with fmaxf), and a
// max of -0 or +0 gives the same exponentials.
struct OpMax {
    __device__ __forceinline__ static float f(float a, float b) { return __builtin_elementwise_maximum(a, b); }
};
struct OpAdd {
    __device__ __forceinline__ static float f(float a, float b) { return a + b; }
};

// Reduction over aligned groups of G lanes; all lanes of a group end with identical bits.
template <int G, class Op>
__device__ __forceinline__ float group_reduce(float v) {
    static_assert(G == 8 || G == 16 || G == 32 || G == 64, "group size");
    v = Op::f(v, dpp<0xB1>(v));   // quad_perm [1,0,3,2]: partner lane ^ 1
    v = Op::f(v, dpp<0x4E>(v));   // quad_perm [2,3,0,1]: partner lane ^ 2
    v = Op::f(v, dpp<0x141>(v));  // row_half_mirror: partner in the other quad of 8
    if constexpr (G >= 16)
        v = Op::f(v, dpp<0x140>(v));  // row_mirror: partner in the other half of the 16-lane row
    if constexpr (G >= 32) {      // rows 2k and 2k+1 meet
        auto p = __builtin_amdgcn_permlane16_swap(f_bits(v), f_bits(v), false, false);
        v = Op::f(bits_f(p[0]), bits_f(p[1]));
    }
    if constexpr (G == 64) {      // the two 32-lane halves meet
        auto p = __builtin_amdgcn_permlane32_swap(f_bits(v), f_bits(v), false, false);
        v = Op::f(bits_f(p[0]), bits_f(p[1]));
    }
    return v;
}

// In-lane pairwise reduction of K values: neighbours combine in pairs, an odd last value is
// carried to the next level, until one is left (a fixed tree for each K).
template <int K, class Op>
__device__ __forceinline__ float lane_reduce(const float* x) {
    static_assert(K > 0, "lane_reduce needs a value");
    if constexpr (K == 1) {
        return x[0];
    } else {
        constexpr int H = (K + 1) / 2;
        float t[H];
#pragma unroll
        for (int i = 0; i < K / 2; ++i) t[i] = Op::f(x[2 * i], x[2 * i + 1]);
        if constexpr (K % 2 == 1) t[H - 1] = x[K - 1];
        return lane_reduce<H, Op>(t);
    }
}

// In-lane sum of a[k] g[k] by the same pairwise tree, its first level fused: a[2i] g[2i] +
// a[2i+1] g[2i+1] as one fma over one product, so that no product is held in a register of its
// own (with K products formed first, a backward row held by a lane needs 3K values at once).
template <int K>
__device__ __forceinline__ float lane_dot(const float* a, const float* g) {
    static_assert(K > 0, "lane_dot needs a value");
    if constexpr (K == 1) {
        return a[0] * g[0];
    } else {
        constexpr int H = (K + 1) / 2;
        float t[H];
#pragma unroll
        for (int i = 0; i < K / 2; ++i) t[i] = __builtin_fmaf(a[2 * i], g[2 * i], a[2 * i + 1] * g[2 * i + 1]);
        if constexpr (K % 2 == 1) t[H - 1] = a[K - 1] * g[K - 1];
        return lane_reduce<H, OpAdd>(t);
    }
}

// 16-byte accesses, nontemporal (streaming) or ordinary (cache-resident) by NT.
template <bool NT, class V>
__device__ __forceinline__ V load16(const V* p) {
    if constexpr (NT) return __builtin_nontemporal_load(p);
    return *p;
}
template <bool NT, class V>
__device__ __forceinline__ void store16(V* p, V v) {
    if constexpr (NT) __builtin_nontemporal_store(v, p);
    else *p = v;
}

template <bool NT>
struct F32 {
    using T = float;
    static constexpr int kBytes = 4;
    static constexpr int kEPV = 4;  // elements per 16-byte vector
    using R = f32x4;  // one 16-byte vector as loaded
    __device__ __forceinline__ static R load_raw(const T* p) { return load16<NT>(reinterpret_cast<const R*>(p)); }
    __device__ __forceinline__ static R raw_fill(float f) { return R{f, f, f, f}; }
    __device__ __forceinline__ static void unpack(R v, float* x) {
        x[0] = v.x; x[1] = v.y; x[2] = v.z; x[3] = v.w;
    }
    __device__ __forceinline__ static void load_vec(const T* p, float* x) { unpack(load_raw(p), x); }
    __device__ __forceinline__ static void store_vec(T* p, const float* y) {
        store16<NT>(reinterpret_cast<f32x4*>(p), f32x4{y[0], y[1], y[2], y[3]});
    }
    __device__ __forceinline__ static float load1(const T* p) { return *p; }
    __device__ __forceinline__ static void store1(T* p, float y) { *p = y; }
};

template <bool NT>
struct BF16 {
    using T = uint16_t;  // raw bf16 bit pattern
    static constexpr int kBytes = 2;
    static constexpr int kEPV = 8;
    using R = u32x4;  // one 16-byte vector as loaded: eight bf16 bit patterns
    __device__ __forceinline__ static R load_raw(const T* p) { return load16<NT>(reinterpret_cast<const R*>(p)); }
    // f's bf16 pattern twice per dword (exact for the fills used: -inf and 0)
    __device__ __forceinline__ static R raw_fill(float f) {
        const unsigned h = f_bits(f) >> 16;
        return R{h | (h << 16), h | (h << 16), h | (h << 16), h | (h << 16)};
    }
    __device__ __forceinline__ static void unpack(R v, float* x) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            x[2 * i] = bits_f(v[i] << 16);
            x[2 * i + 1] = bits_f(v[i] & 0xFFFF0000u);
        }
    }
    __device__ __forceinline__ static void load_vec(const T* p, float* x) { unpack(load_raw(p), x); }
    __device__ __forceinline__ static unsigned pack(float a, float b) {
        // round to nearest even, NaN stays NaN (v_cvt_pk_bf16_f32)
        return __builtin_bit_cast(unsigned, __builtin_convertvector(f32x2{a, b}, bf16x2));
    }
    __device__ __forceinline__ static void store_vec(T* p, const float* y) {
        store16<NT>(reinterpret_cast<u32x4*>(p),
                    u32x4{pack(y[0], y[1]), pack(y[2], y[3]), pack(y[4], y[5]), pack(y[6], y[7])});
    }
    __device__ __forceinline__ static float load1(const T* p) {
        return bits_f(static_cast<unsigned>(*p) << 16);
    }
    __device__ __forceinline__ static void store1(T* p, float y) {
        *p = __builtin_bit_cast(uint16_t, static_cast<__bf16>(y));
    }
};

// Softmax of U rows per group, all loads first (U rows x V vectors in flight per lane).
//   row r of the item starts at element base + r * cols; rows r0, r0 + step, ...
// The 16-byte vectors of one row.  An aligned row (SHIFT false: its start and length whole
// vectors) holds cols / EPV of them from its start.  A shifted row -- start or length not a
// whole number of vectors, the buffers themselves 16-byte aligned -- is covered by the aligned
// vectors from the one holding its first element: the first `ph` elements of vector 0 precede
// the row and the last vector may run past its end.  Those outside elements are read with the
// vector (a 16-byte vector never crosses a page, so it is mapped wherever one of its elements
// is) and replaced by `pad`, and never written: the row's first and last vectors are stored
// element by element, every other one as a whole.
template <class E, bool SHIFT>
struct RowVecs {
    static constexpr int EPV = E::kEPV;
    int64_t start;  // element offset of vector 0
    int ph;         // elements of vector 0 before the row
    int cols;
    int nv;         // vectors covering the row
    __device__ __forceinline__ RowVecs(int64_t row_start, int c) : cols(c) {
        ph = SHIFT ? static_cast<int>(row_start & (EPV - 1)) : 0;
        start = row_start - ph;
        nv = SHIFT ? (ph + c + EPV - 1) / EPV : c / EPV;
    }
    // Elements [lo, hi) of vector vi belong to the row.
    __device__ __forceinline__ int lo(int vi) const { return ph - vi * EPV; }
    __device__ __forceinline__ int hi(int vi) const { return cols + ph - vi * EPV; }
    __device__ __forceinline__ void mask(int vi, float* x, float pad) const {
        if constexpr (SHIFT) {
            const int l = lo(vi), h = hi(vi);
            if (l > 0 || h < EPV) {
#pragma unroll
                for (int e = 0; e < EPV; ++e)
                    if (e < l || e >= h) x[e] = pad;
            }
        }
    }
    __device__ __forceinline__ void store(typename E::T* out, int vi, const float* y) const {
        typename E::T* p = out + start + vi * EPV;
        if constexpr (SHIFT) {
            const int l = lo(vi), h = hi(vi);
            if (l > 0 || h < EPV) {
#pragma unroll
                for (int e = 0; e < EPV; ++e)
                    if (e >= l && e < h) E::store1(p + e, y[e]);
                return;
            }
        }
        E::store_vec(p, y);
    }
};

// Vectors a row of `cols` elements may span: one more than its length in vectors when shifted.
template <class E, bool SHIFT>
__device__ __forceinline__ int span_vecs(int cols) {
    return (cols + E::kEPV - 1) / E::kEPV + (SHIFT ? 1 : 0);
}

template <class E, int G, int V, int U, bool VEC, bool SHIFT = false>
__device__ __forceinline__ void rows_u(const typename E::T* in, typename E::T* out, int64_t base,
                                       int cols, int nrows, int r0, int step, int lane) {
    constexpr int EPV = E::kEPV;
    constexpr int K = V * EPV;
    float x[U][K];
    typename E::R raw[U][V];
    bool act[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int r = r0 + u * step;
        act[u] = r < nrows;
        const int64_t o = base + static_cast<int64_t>(r) * cols;
        if constexpr (VEC) {
            // the vectors as loaded (a lane's loads all issued before any use; unpacking
            // inside each conditional load would make every load wait for the previous one)
            const RowVecs<E, SHIFT> rv(o, cols);
#pragma unroll
            for (int v = 0; v < V; ++v) {
                const int vi = lane + v * G;
                if (act[u] && vi < rv.nv)
                    raw[u][v] = E::load_raw(in + rv.start + vi * EPV);
                else
                    raw[u][v] = E::raw_fill(kNegInf);
            }
        } else {
#pragma unroll
            for (int k = 0; k < K; ++k) {
                const int j = lane + k * G;
                x[u][k] = (act[u] && j < cols) ? E::load1(in + o + j) : kNegInf;
            }
        }
    }
    if constexpr (VEC) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const RowVecs<E, SHIFT> rv(base + static_cast<int64_t>(r0 + u * step) * cols, cols);
#pragma unroll
            for (int v = 0; v < V; ++v) {
                E::unpack(raw[u][v], &x[u][v * EPV]);
                rv.mask(lane + v * G, &x[u][v * EPV], kNegInf);
            }
        }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
        float m = group_reduce<G, OpMax>(lane_reduce<K, OpMax>(x[u]));
        const float ms = (m == kNegInf) ? 0.0f : m;  // fully masked row: every e is 0
#pragma unroll
        for (int k = 0; k < K; ++k) x[u][k] = __builtin_amdgcn_exp2f((x[u][k] - ms) * kLog2e);
        const float s = group_reduce<G, OpAdd>(lane_reduce<K, OpAdd>(x[u]));
        const float inv = (s == 0.0f) ? 0.0f : __builtin_amdgcn_rcpf(s);
#pragma unroll
        for (int k = 0; k < K; ++k) x[u][k] *= inv;
        const int r = r0 + u * step;
        const int64_t o = base + static_cast<int64_t>(r) * cols;
        if constexpr (VEC) {
            const RowVecs<E, SHIFT> rv(o, cols);
#pragma unroll
            for (int v = 0; v < V; ++v) {
                const int vi = lane + v * G;
                if (act[u] && vi < rv.nv) rv.store(out, vi, &x[u][v * EPV]);
            }
        } else {
#pragma unroll
            for (int k = 0; k < K; ++k) {
                const int j = lane + k * G;
                if (act[u] && j < cols) E::store1(out + o + j, x[u][k]);
            }
        }
    }
}

// The reductions of U rows held by lanes gb .. gb + n - 1 each (n <= 32, any n; i = lane - gb):
// a tree to the row's first lane (lane i < d takes lane i + d while i + d < n, d = 16, 8, 4, 2,
// 1), then one ds_bpermute from it, so every lane of a row ends with the same bits.  Each step
// is taken for all U rows before the next, so that their LDS round trips overlap.
template <class Op, int U>
__device__ __forceinline__ void seg_reduce(float (&a)[U], int i, int n, int gb) {
#pragma unroll
    for (int d = 16; d >= 1; d /= 2) {
        float o[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            o[u] = __builtin_bit_cast(
                float, __builtin_amdgcn_ds_bpermute((gb + i + d) << 2, __builtin_bit_cast(int, a[u])));
        const bool take = i < d && i + d < n;
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (take) a[u] = Op::f(a[u], o[u]);
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
        a[u] = __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute(gb << 2, __builtin_bit_cast(int, a[u])));
}

// Packed tile (tile_for's G = n, not a power of two): aligned rows of n vectors, 64 / n rows side
// by side in a wave, row g on lanes [g n, g n + n), one vector per lane, U rows per group in
// flight.  A load instruction then moves 64 / n consecutive rows with almost every lane busy,
// where a power-of-two group would leave up to half of its lanes idle.
template <class E, int U>
__device__ __forceinline__ void rows_packed(const typename E::T* in, typename E::T* out,
                                            int64_t base, int n, int nrows, int r0, int step,
                                            int i, int gb, bool on) {
    constexpr int EPV = E::kEPV;
    const int cols = n * EPV;
    float x[U][EPV];
    typename E::R raw[U];
    bool act[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int r = r0 + u * step;
        act[u] = on && r < nrows;
        raw[u] = act[u] ? E::load_raw(in + base + static_cast<int64_t>(r) * cols + i * EPV)
                        : E::raw_fill(kNegInf);
    }
    float m[U], s[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        E::unpack(raw[u], x[u]);
        m[u] = lane_reduce<EPV, OpMax>(x[u]);
    }
    seg_reduce<OpMax, U>(m, i, n, gb);
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const float ms = (m[u] == kNegInf) ? 0.0f : m[u];
#pragma unroll
        for (int k = 0; k < EPV; ++k) x[u][k] = __builtin_amdgcn_exp2f((x[u][k] - ms) * kLog2e);
        s[u] = lane_reduce<EPV, OpAdd>(x[u]);
    }
    seg_reduce<OpAdd, U>(s, i, n, gb);
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const float inv = (s[u] == 0.0f) ? 0.0f : __builtin_amdgcn_rcpf(s[u]);
#pragma unroll
        for (int k = 0; k < EPV; ++k) x[u][k] *= inv;
        if (act[u])
            E::store_vec(out + base + static_cast<int64_t>(r0 + u * step) * cols + i * EPV, x[u]);
    }
}

// One item in packed tiles, walked like run_item with 64 / n rows per wave.
template <class E, int U>
__device__ __forceinline__ uint32_t run_item_packed(const typename E::T* in, typename E::T* out,
                                                    int64_t base, int cols, int nrows, int reps,
                                                    int64_t stride, int wave, int nwaves,
                                                    int lane64) {
    const int n = cols / E::kEPV;
    const int rpw = 64 / n;
    const int sub = lane64 / n;
    const int i = lane64 - sub * n;
    const bool on = sub < rpw;
    const int gb = sub * n;
    const int step = nwaves * rpw;
    uint32_t done = 0;
    for (int k = 0; k < reps; ++k) {
        const int64_t b = base + k * stride;
        int r0 = wave * rpw;
        for (; r0 + (U - 1) * step < nrows; r0 += U * step) {
            rows_packed<E, U>(in, out, b, n, nrows, r0 + sub, step, i, gb, on);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int left = nrows - (r0 + u * step);
                done += left < rpw ? left : rpw;
            }
        }
        for (; r0 < nrows; r0 += step) {
            rows_packed<E, 1>(in, out, b, n, nrows, r0 + sub, step, i, gb, on);
            const int left = nrows - r0;
            done += left < rpw ? left : rpw;
        }
    }
    return done;
}

// One item with G lanes per row: `reps` ranges of `nrows` rows, range k starting at element
// base + k * stride.  Within a range the worker's rows are wave*RPW + sub + j*step, j = 0, 1,
// ... (RPW = 64/G rows per wave, step = rows covered by all the worker's waves at once); loop
// trip counts depend on the wave only, so lanes never diverge across iterations.
template <class E, int G, int V, int U, bool VEC, bool SHIFT>
__device__ __forceinline__ uint32_t run_item(const typename E::T* in, typename E::T* out,
                                             int64_t base, int cols, int nrows, int reps,
                                             int64_t stride, int wave, int nwaves, int lane64) {
    constexpr int RPW = 64 / G;
    const int sub = lane64 / G;
    const int lane = lane64 % G;
    const int step = nwaves * RPW;
    uint32_t done = 0;
    for (int k = 0; k < reps; ++k) {
        const int64_t b = base + k * stride;
        int r0 = wave * RPW;
        // U rows per group while the last of them still has a row; the rest one at a time, so a
        // short remainder does not pay for U rows
        for (; r0 + (U - 1) * step < nrows; r0 += U * step) {
            rows_u<E, G, V, U, VEC, SHIFT>(in, out, b, cols, nrows, r0 + sub, step, lane);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int left = nrows - (r0 + u * step);
                done += left < RPW ? left : RPW;
            }
        }
        if constexpr (U > 1) {
            for (; r0 < nrows; r0 += step) {
                rows_u<E, G, V, 1, VEC, SHIFT>(in, out, b, cols, nrows, r0 + sub, step, lane);
                const int left = nrows - r0;
                done += left < RPW ? left : RPW;
            }
        }
    }
    return done;
}

// One wave per row, for rows that neither a register tile nor the workgroup path takes: rows
// whose start or length is not 16-byte aligned, beyond 64 vectors (element-wise, in chunks of
// 8 elements, whose per-element addresses cost registers), and in the backward pass aligned
// rows of 257..512 vectors (chunks of CH 16-byte vectors per lane, VALS values: 32 for one
// input stream, 16 for two, so each lane keeps CH loads in flight).
//
// When the row fits the wave's LDS region (`cap` floats, given to plans with long rows), it is
// read from HBM once: pass 1 keeps a per-lane max while staging the values in LDS, pass 2
// turns the staged values into e = 2^((x - M) log2 e) in place and sums them, pass 3 writes
// e * (1/S).  Every lane re-reads only what it wrote itself, so no barrier is needed.
//
// Otherwise two passes over HBM: pass 1 keeps a per-lane running max and a sum rescaled
// whenever a chunk raises the max, the lanes' pairs are merged, pass 2 re-reads the row and
// writes e * (1/S) (1.5x the bytes of the staged path).
template <class E, bool VEC, int VALS = 32>
struct LongRow {
    using T = typename E::T;
    static constexpr int EPV = E::kEPV;
    static constexpr int CH = VALS / EPV;      // vectors per lane per chunk (aligned rows)
    static constexpr int K = VEC ? CH * EPV : 8;  // values per lane per chunk

    // Loads chunk c0 (vector index of the lane's first vector, stride 64) into x; vectors past
    // the row are -inf.  Element-wise variant: elements j0 + 64 k.
    __device__ __forceinline__ static void load(const T* src, int cols, int first, float* x,
                                                float pad = kNegInf) {
        if constexpr (VEC) {
            // every load of the chunk issued before any is unpacked (as in rows_u)
            const int nvec = cols / EPV;
            typename E::R raw[CH];
#pragma unroll
            for (int c = 0; c < CH; ++c) {
                const int vi = first + c * 64;
                if (vi < nvec)
                    raw[c] = E::load_raw(src + vi * EPV);
                else
                    raw[c] = E::raw_fill(pad);
            }
#pragma unroll
            for (int c = 0; c < CH; ++c) E::unpack(raw[c], x + c * EPV);
        } else {
#pragma unroll
            for (int k = 0; k < K; ++k) {
                const int j = first + k * 64;
                x[k] = j < cols ? E::load1(src + j) : pad;
            }
        }
    }
    // The lane's values of a chunk to / from LDS at their element index (each lane touches
    // only what it wrote itself).
    __device__ __forceinline__ static void to_lds(float* lds, int cols, int first, const float* x) {
        if constexpr (VEC) {
            const int nvec = cols / EPV;
#pragma unroll
            for (int c = 0; c < CH; ++c) {
                const int vi = first + c * 64;
                if (vi < nvec) {
#pragma unroll
                    for (int i = 0; i < EPV; i += 4)
                        *reinterpret_cast<f32x4*>(lds + vi * EPV + i) =
                            f32x4{x[c * EPV + i], x[c * EPV + i + 1], x[c * EPV + i + 2], x[c * EPV + i + 3]};
                }
            }
        } else {
#pragma unroll
            for (int k = 0; k < K; ++k) {
                const int j = first + k * 64;
                if (j < cols) lds[j] = x[k];
            }
        }
    }
    __device__ __forceinline__ static void from_lds(const float* lds, int cols, int first, float* x,
                                                    float pad) {
        if constexpr (VEC) {
            const int nvec = cols / EPV;
#pragma unroll
            for (int c = 0; c < CH; ++c) {
                const int vi = first + c * 64;
#pragma unroll
                for (int i = 0; i < EPV; i += 4) {
                    f32x4 v = f32x4{pad, pad, pad, pad};
                    if (vi < nvec) v = *reinterpret_cast<const f32x4*>(lds + vi * EPV + i);
                    x[c * EPV + i] = v.x;
                    x[c * EPV + i + 1] = v.y;
                    x[c * EPV + i + 2] = v.z;
                    x[c * EPV + i + 3] = v.w;
                }
            }
        } else {
#pragma unroll
            for (int k = 0; k < K; ++k) {
                const int j = first + k * 64;
                x[k] = j < cols ? lds[j] : pad;
            }
        }
    }
    __device__ __forceinline__ static void store(T* dst, int cols, int first, const float* y) {
        if constexpr (VEC) {
            const int nvec = cols / EPV;
#pragma unroll
            for (int c = 0; c < CH; ++c) {
                const int vi = first + c * 64;
                if (vi < nvec) E::store_vec(dst + vi * EPV, y + c * EPV);
            }
        } else {
#pragma unroll
            for (int k = 0; k < K; ++k) {
                const int j = first + k * 64;
                if (j < cols) E::store1(dst + j, y[k]);
            }
        }
    }
    static constexpr int kStep = VEC ? CH * 64 : K * 64;
    __device__ __forceinline__ static int extent(int cols) { return VEC ? cols / EPV : cols; }
};

// Forward one-wave path: element by element (rows in buffers that are not 16-byte aligned;
// aligned buffers take the register tiles, shifted vectors or the workgroup path).
template <class E, bool STAGE>
__device__ __forceinline__ void long_row(const typename E::T* src, typename E::T* dst, int cols,
                                         int lane, float* lds, int cap) {
    using L = LongRow<E, false>;
    constexpr int K = L::K;
    const int step = L::kStep;
    if (STAGE && cols <= cap) {
        // LDS holds the row as floats at their element index
        float m = kNegInf;
        for (int first = lane; first < cols; first += step) {
            float x[K];
            L::load(src, cols, first, x);
            m = OpMax::f(m, lane_reduce<K, OpMax>(x));
            L::to_lds(lds, cols, first, x);
        }
        const float M = group_reduce<64, OpMax>(m);
        const float Ms = (M == kNegInf) ? 0.0f : M;
        float s = 0.0f;
        for (int first = lane; first < cols; first += step) {
            float e[K];
#pragma unroll
            for (int k = 0; k < K; ++k) {
                const int j = first + k * 64;
                e[k] = j < cols ? __builtin_amdgcn_exp2f((lds[j] - Ms) * kLog2e) : 0.0f;
                if (j < cols) lds[j] = e[k];
            }
            s += lane_reduce<K, OpAdd>(e);
        }
        const float S = group_reduce<64, OpAdd>(s);
        const float inv = (S == 0.0f) ? 0.0f : __builtin_amdgcn_rcpf(S);
        for (int first = lane; first < cols; first += step) {
            float y[K];
            L::from_lds(lds, cols, first, y, 0.0f);
#pragma unroll
            for (int k = 0; k < K; ++k) y[k] *= inv;
            L::store(dst, cols, first, y);
        }
        return;
    }
    float m = kNegInf, s = 0.0f;
    for (int first = lane; first < cols; first += step) {
        float x[K];
        L::load(src, cols, first, x);
        const float cm = lane_reduce<K, OpMax>(x);
        if (cm > m) {
            s *= __builtin_amdgcn_exp2f((m - cm) * kLog2e);
            m = cm;
        }
        if (m != kNegInf) {
#pragma unroll
            for (int k = 0; k < K; ++k) x[k] = __builtin_amdgcn_exp2f((x[k] - m) * kLog2e);
            s += lane_reduce<K, OpAdd>(x);
        }
    }
    const float M = group_reduce<64, OpMax>(m);
    const float Ms = (M == kNegInf) ? 0.0f : M;
    const float scale = (m == kNegInf) ? 0.0f : __builtin_amdgcn_exp2f((m - Ms) * kLog2e);
    const float S = group_reduce<64, OpAdd>(s * scale);
    const float inv = (S == 0.0f) ? 0.0f : __builtin_amdgcn_rcpf(S);
    for (int first = lane; first < cols; first += step) {
        float x[K];
        L::load(src, cols, first, x);
#pragma unroll
        for (int k = 0; k < K; ++k) x[k] = __builtin_amdgcn_exp2f((x[k] - Ms) * kLog2e) * inv;
        L::store(dst, cols, first, x);
    }
}

// ------------------------------------------------------------------------ workgroup rows
// Aligned rows beyond the register tile, one row at a time per workgroup: all of its
// nt = 64 * nwaves lanes share the row, lane t holding vectors t, t + nt, ..., t + (L-1) nt (so
// each load instruction of a wave covers 1 KiB of consecutive bytes).  The row is read once
// into registers; max and sum are the in-lane tree, the wave's butterfly, then the waves'
// values combined in wave order through LDS (two barriers per row), so every lane of the
// workgroup ends with the same bits and a row's result depends on its values, its length and
// the workgroup size only.  Rows beyond L vectors per lane take two passes over HBM with a
// per-lane running max and rescaled sum (as in long_row), combined the same way.
constexpr int kTeamMaxRows = 2;  // rows a workgroup keeps in flight
__shared__ float team_slots[2][kTeamMaxRows][16];  // [max, sum][row][wave]: lane 0 of each wave

// Combine U values per wave (one per row) in wave order; slot set `which` is reused by the next
// rows only after the other set's barrier, which every wave reaches after reading this one.
template <class Op, int U>
__device__ __forceinline__ void team_combine(float (&v)[U], int which, int wave, int nwaves,
                                             int lane) {
    if (lane == 0) {
#pragma unroll
        for (int u = 0; u < U; ++u) team_slots[which][u][wave] = v[u];
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < U; ++u) {
        float r = team_slots[which][u][0];
        for (int i = 1; i < nwaves; ++i) r = Op::f(r, team_slots[which][u][i]);
        v[u] = r;
    }
}

// Lane t's vectors t + c nt, c < L, of row rv; vectors past the row (or of an inactive row)
// read as `pad`, and so do a shifted row's outside elements (after team_unpack).
template <class E, int L, bool SHIFT>
__device__ __forceinline__ void team_load(const typename E::T* in, const RowVecs<E, SHIFT>& rv,
                                          int first, int nt, bool act, typename E::R* raw,
                                          float pad = kNegInf) {
    constexpr int EPV = E::kEPV;
#pragma unroll
    for (int c = 0; c < L; ++c) {
        const int vi = first + c * nt;
        raw[c] = (act && vi < rv.nv) ? E::load_raw(in + rv.start + vi * EPV) : E::raw_fill(pad);
    }
}

template <class E, int L, bool SHIFT>
__device__ __forceinline__ void team_unpack(const RowVecs<E, SHIFT>& rv, int first, int nt,
                                            const typename E::R* raw, float* x,
                                            float pad = kNegInf) {
#pragma unroll
    for (int c = 0; c < L; ++c) {
        E::unpack(raw[c], x + c * E::kEPV);
        rv.mask(first + c * nt, x + c * E::kEPV, pad);
    }
}

template <class E, int L, bool SHIFT>
__device__ __forceinline__ void team_store(typename E::T* out, const RowVecs<E, SHIFT>& rv,
                                           int first, int nt, bool act, const float* y) {
#pragma unroll
    for (int c = 0; c < L; ++c) {
        const int vi = first + c * nt;
        if (act && vi < rv.nv) rv.store(out, vi, y + c * E::kEPV);
    }
}

// Up to U rows (those with act[u], starting at elements off[u]) held in registers: L vectors
// per lane cover nt * L vectors of a row.  A row's arithmetic does not depend on U.
template <class E, int L, int U, bool SHIFT>
__device__ __forceinline__ void team_rows(const typename E::T* in, typename E::T* out,
                                          const int64_t (&off)[U], const bool (&act)[U], int cols,
                                          int t, int nt, int wave, int nwaves, int lane) {
    constexpr int K = L * E::kEPV;
    float x[U][K];
    typename E::R raw[U][L];
#pragma unroll
    for (int u = 0; u < U; ++u)
        team_load<E, L, SHIFT>(in, RowVecs<E, SHIFT>(off[u], cols), t, nt, act[u], raw[u]);
#pragma unroll
    for (int u = 0; u < U; ++u)
        team_unpack<E, L, SHIFT>(RowVecs<E, SHIFT>(off[u], cols), t, nt, raw[u], x[u]);
    float m[U];
#pragma unroll
    for (int u = 0; u < U; ++u) m[u] = group_reduce<64, OpMax>(lane_reduce<K, OpMax>(x[u]));
    team_combine<OpMax, U>(m, 0, wave, nwaves, lane);
    float s[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const float ms = (m[u] == kNegInf) ? 0.0f : m[u];
#pragma unroll
        for (int k = 0; k < K; ++k) x[u][k] = __builtin_amdgcn_exp2f((x[u][k] - ms) * kLog2e);
        s[u] = group_reduce<64, OpAdd>(lane_reduce<K, OpAdd>(x[u]));
    }
    team_combine<OpAdd, U>(s, 1, wave, nwaves, lane);
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const float inv = (s[u] == 0.0f) ? 0.0f : __builtin_amdgcn_rcpf(s[u]);
#pragma unroll
        for (int k = 0; k < K; ++k) x[u][k] *= inv;
        team_store<E, L, SHIFT>(out, RowVecs<E, SHIFT>(off[u], cols), t, nt, act[u], x[u]);
    }
}

// The trace counts row j of an item's sequence for wave j mod nwaves.
__device__ __forceinline__ uint32_t team_rows_of_wave(int nrows, int reps, int wave, int nwaves) {
    const int64_t total = static_cast<int64_t>(nrows) * reps;
    return total > wave ? static_cast<uint32_t>((total - wave + nwaves - 1) / nwaves) : 0u;
}

template <int U>
struct RowWalk {
    int64_t base, stride, total, j = 0;
    int cols, nrows, k = 0, r = 0;
    __device__ RowWalk(int64_t b, int c, int n, int reps, int64_t st)
        : base(b), stride(st), total(static_cast<int64_t>(n) * reps), cols(c), nrows(n) {}
    __device__ bool more() const { return j < total; }
    __device__ void next(int64_t (&off)[U], bool (&act)[U]) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            act[u] = j < total;
            off[u] = base + k * stride + static_cast<int64_t>(r) * cols;
            if (act[u]) {
                ++j;
                if (++r == nrows) {
                    r = 0;
                    ++k;
                }
            }
        }
    }
};

// A row longer than nt * L vectors: chunks of nt * L vectors, read twice.
template <class E, int L, bool SHIFT>
__device__ __forceinline__ void team_row_two_pass(const typename E::T* in, typename E::T* out,
                                                  int64_t off, int cols, int t, int nt, int wave,
                                                  int nwaves, int lane) {
    constexpr int K = L * E::kEPV;
    const RowVecs<E, SHIFT> rv(off, cols);
    float m = kNegInf, s = 0.0f;
    for (int first = t; first - t < rv.nv; first += nt * L) {
        float x[K];
        typename E::R raw[L];
        team_load<E, L, SHIFT>(in, rv, first, nt, true, raw);
        team_unpack<E, L, SHIFT>(rv, first, nt, raw, x);
        const float cm = lane_reduce<K, OpMax>(x);
        if (cm > m) {
            s *= __builtin_amdgcn_exp2f((m - cm) * kLog2e);
            m = cm;
        }
        if (m != kNegInf) {
#pragma unroll
            for (int k = 0; k < K; ++k) x[k] = __builtin_amdgcn_exp2f((x[k] - m) * kLog2e);
            s += lane_reduce<K, OpAdd>(x);
        }
    }
    float M[1] = {group_reduce<64, OpMax>(m)};
    team_combine<OpMax, 1>(M, 0, wave, nwaves, lane);
    const float Ms = (M[0] == kNegInf) ? 0.0f : M[0];
    const float scale = (m == kNegInf) ? 0.0f : __builtin_amdgcn_exp2f((m - Ms) * kLog2e);
    float S[1] = {group_reduce<64, OpAdd>(s * scale)};
    team_combine<OpAdd, 1>(S, 1, wave, nwaves, lane);
    const float inv = (S[0] == 0.0f) ? 0.0f : __builtin_amdgcn_rcpf(S[0]);
    for (int first = t; first - t < rv.nv; first += nt * L) {
        float x[K];
        typename E::R raw[L];
        team_load<E, L, SHIFT>(in, rv, first, nt, true, raw);
        team_unpack<E, L, SHIFT>(rv, first, nt, raw, x);
#pragma unroll
        for (int k = 0; k < K; ++k) x[k] = __builtin_amdgcn_exp2f((x[k] - Ms) * kLog2e) * inv;
        team_store<E, L, SHIFT>(out, rv, first, nt, true, x);
    }
}

// Vectors per lane (and per input stream) of a register-held row: bsm::kTeamValues values per
// lane in kernel class 4, twice that in class 5.
template <class E, int KCLASS>
constexpr int kTeamMaxL = (KCLASS >= 5 ? 2 : 1) * bsm::kTeamValues / E::kEPV;  // 6 as 5

// Every row of an item, each by the whole workgroup.  The trace counts row r for wave
// r mod nwaves.
template <class E, int KCLASS, bool SHIFT>
__device__ __forceinline__ uint32_t team_item(const typename E::T* in, typename E::T* out,
                                              int64_t base, int cols, int nrows, int reps,
                                              int64_t stride, int wave, int nwaves, int lane) {
    const int nt = nwaves * 64;
    const int t = wave * 64 + lane;
    const int per_lane = (span_vecs<E, SHIFT>(cols) + nt - 1) / nt;
    constexpr int kMaxL = kTeamMaxL<E, KCLASS>;  // 4 or 8 (class 4), 8 or 16 (class 5)
    if (per_lane <= 3) {
        // the shortest rows (at most 3 of the 4 vectors per lane): two in flight, so that a lane
        // keeps 5-6 loads outstanding (measured: 2500-element fp32 rows 5.7 TB/s against 4.9 one
        // at a time; rows filling 4 vectors per lane are 2% faster one at a time)
        RowWalk<2> w(base, cols, nrows, reps, stride);
        while (w.more()) {
            int64_t off[2];
            bool act[2];
            w.next(off, act);
            team_rows<E, 4, 2, SHIFT>(in, out, off, act, cols, t, nt, wave, nwaves, lane);
        }
    } else if (E::kBytes == 2 && kMaxL >= 6 && per_lane <= 6) {
        // bf16 rows of 5 or 6 vectors per lane (e.g. 8200 elements): two rows in flight, as for
        // the shortest rows (8200 bf16: 4.05 -> 4.3 TB/s against one row of 8 vectors per lane,
        // 5 of them used; fp32 rows lost 1.5-4% this way and keep one row of 8), in a tile of
        // exactly 5 slots where 5 suffice (8200 bf16: 4.76 -> 4.97 TB/s against 6; the
        // backward pass lost 5% with a 5-slot tile and keeps its 8)
        RowWalk<2> w(base, cols, nrows, reps, stride);
        while (w.more()) {
            int64_t off[2];
            bool act[2];
            w.next(off, act);
            if (per_lane <= 5)
                team_rows<E, (kMaxL >= 6 ? 5 : 4), 2, SHIFT>(in, out, off, act, cols, t, nt, wave,
                                                             nwaves, lane);
            else
                team_rows<E, (kMaxL >= 6 ? 6 : 4), 2, SHIFT>(in, out, off, act, cols, t, nt, wave,
                                                             nwaves, lane);
        }
    } else if (per_lane <= kMaxL) {
        RowWalk<1> w(base, cols, nrows, reps, stride);
        while (w.more()) {
            int64_t off[1];
            bool act[1];
            w.next(off, act);
            if (per_lane <= 4)
                team_rows<E, 4, 1, SHIFT>(in, out, off, act, cols, t, nt, wave, nwaves, lane);
            else if (kMaxL > 8 && per_lane <= 8)
                team_rows<E, (kMaxL > 8 ? 8 : kMaxL), 1, SHIFT>(in, out, off, act, cols, t, nt,
                                                                wave, nwaves, lane);
            else
                team_rows<E, kMaxL, 1, SHIFT>(in, out, off, act, cols, t, nt, wave, nwaves, lane);
        }
    } else {
        RowWalk<1> w(base, cols, nrows, reps, stride);
        while (w.more()) {
            int64_t off[1];
            bool act[1];
            w.next(off, act);
            team_row_two_pass<E, kMaxL, SHIFT>(in, out, off[0], cols, t, nt, wave, nwaves, lane);
        }
    }
    return team_rows_of_wave(nrows, reps, wave, nwaves);
}

// Vectors the largest register tile of a kernel class covers (classes 4 and 5: any row).
template <int KCLASS>
constexpr int kClassMaxVecs = KCLASS == 0 ? 64 : KCLASS == 1 ? 128 : KCLASS == 2 ? 256
                              : KCLASS == 3 ? 512 : 0x7FFFFFFF;

// Register-tile choice per item (wave-uniform branch); the thresholds are bsm::tile_for's.  A
// shifted item's tile covers the vectors its rows may span (one more than their length).
template <class E, int KCLASS, bool VEC, bool SHIFT>
__device__ __forceinline__ uint32_t dispatch_item(const typename E::T* in, typename E::T* out,
                                                  int64_t base, int cols, int nrows, int reps,
                                                  int64_t stride, int wave, int nwaves,
                                                  int lane64, float* lds, int cap, bool team) {
    const int nvec = VEC ? span_vecs<E, SHIFT>(cols) : (cols + E::kEPV - 1) / E::kEPV;
#define BSM_RUN(G, V, U) run_item<E, G, V, U, VEC, SHIFT>(in, out, base, cols, nrows, reps, stride, wave, nwaves, lane64)
    if constexpr (VEC) {
        // the tile of bsm::tile_for: one wave-uniform branch per (G, V, U) the class can pick
        constexpr bool F = E::kBytes == 4;
        const bsm::Tile t = bsm::tile_for(nvec, KCLASS < 4 ? KCLASS : 4, E::kBytes, !SHIFT);
        if constexpr (!SHIFT && KCLASS == 0) {
            if (t.V == 1 && (t.G & (t.G - 1)) != 0)  // packed tile
                return run_item_packed<E, 4>(in, out, base, cols, nrows, reps, stride, wave,
                                             nwaves, lane64);
        }
#define BSM_TILE(g, v, u) if (t.G == g && t.V == v && t.U == u) return BSM_RUN(g, v, u)
        if constexpr (KCLASS == 0) BSM_TILE(8, 1, 4);
        BSM_TILE(16, 1, 4);
        if constexpr (F) BSM_TILE(32, 1, 8);
        BSM_TILE(32, 1, 4);
        if constexpr (KCLASS >= 1) {
            if constexpr (F) {
                BSM_TILE(32, 2, 4);
                BSM_TILE(16, 5, 1);
                BSM_TILE(64, 2, 3);
            }
            BSM_TILE(32, 2, 2);
            BSM_TILE(64, 2, 2);
        }
        if constexpr (KCLASS >= 2) {
            if constexpr (F) BSM_TILE(32, 5, 1);
            BSM_TILE(64, 4, 1);
        }
        if constexpr (KCLASS >= 3) {
            if constexpr (F) BSM_TILE(64, 5, 1);
            BSM_TILE(64, 8, 1);
        }
        if constexpr (KCLASS >= 4) {
            BSM_TILE(64, 10, 1);
            BSM_TILE(64, 12, 1);
        }
#undef BSM_TILE
    } else {
        // element-wise rows (buffers not 16-byte aligned), one row per group in flight: the
        // per-element addresses cost registers; longer rows take the one-wave path
        if (nvec <= 16) return BSM_RUN(16, 1, 1);
        if (nvec <= 32) return BSM_RUN(32, 1, 1);
        if (nvec <= 64) return BSM_RUN(64, 1, 1);
    }
#undef BSM_RUN
    if constexpr (VEC && KCLASS >= 4) {
        // the host gives long-row plans workgroup workers (team != 0): the waves share each row
        if (team)
            return team_item<E, KCLASS, SHIFT>(in, out, base, cols, nrows, reps, stride, wave,
                                               nwaves, lane64);
    }
    if constexpr (!VEC || KCLASS >= 4) {
        uint32_t done = 0;
        for (int k = 0; k < reps; ++k) {
            for (int r = wave; r < nrows; r += nwaves) {
                const int64_t o = base + k * stride + static_cast<int64_t>(r) * cols;
                // element by element (an aligned item gets here only in a per-wave table of a
                // long-row class, which the host never builds); only the long-row classes are
                // launched with LDS to stage rows in
                long_row<E, (KCLASS >= 4)>(in + o, out + o, cols, lane64, lds, cap);
                ++done;
            }
        }
        return done;
    }
    return 0;  // unreachable: the item's access path is chosen so that its class covers it
}

// ------------------------------------------------------------------------------- backward
// Gradient of the row softmax (the backward pass of Section 1's batch algorithms): with y the
// forward output and dy the gradient with respect to y, dx = y * (dy - d), d = sum_j dy_j y_j.
// Same register tiles as the forward pass: d is an in-lane pairwise tree of the products, then
// the group's fixed butterfly, so the bits depend on the row's values and length only.  Two
// input streams: half as many rows per group in flight, and tiles up to 4 vectors per lane
// (longer rows take the long-row path).

template <class E, int G, int V, int U, bool VEC, bool SHIFT = false>
__device__ __forceinline__ void rows_u_bwd(const typename E::T* y, const typename E::T* dy,
                                           typename E::T* dx, int64_t base, int cols, int nrows,
                                           int r0, int step, int lane) {
    constexpr int EPV = E::kEPV;
    constexpr int K = V * EPV;
    float a[U][K], g[U][K];
    typename E::R ra[U][V], rg[U][V];
    bool act[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int r = r0 + u * step;
        act[u] = r < nrows;
        const int64_t o = base + static_cast<int64_t>(r) * cols;
        if constexpr (VEC) {
            const RowVecs<E, SHIFT> rv(o, cols);
#pragma unroll
            for (int v = 0; v < V; ++v) {
                const int vi = lane + v * G;
                if (act[u] && vi < rv.nv) {
                    ra[u][v] = E::load_raw(y + rv.start + vi * EPV);
                    rg[u][v] = E::load_raw(dy + rv.start + vi * EPV);
                } else {
                    ra[u][v] = rg[u][v] = E::raw_fill(0.0f);
                }
            }
        } else {
#pragma unroll
            for (int k = 0; k < K; ++k) {
                const int j = lane + k * G;
                const bool in = act[u] && j < cols;
                a[u][k] = in ? E::load1(y + o + j) : 0.0f;
                g[u][k] = in ? E::load1(dy + o + j) : 0.0f;
            }
        }
    }
    if constexpr (VEC) {  // unpacked after every load is issued; outside elements are 0
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const RowVecs<E, SHIFT> rv(base + static_cast<int64_t>(r0 + u * step) * cols, cols);
#pragma unroll
            for (int v = 0; v < V; ++v) {
                E::unpack(ra[u][v], &a[u][v * EPV]);
                E::unpack(rg[u][v], &g[u][v * EPV]);
                rv.mask(lane + v * G, &a[u][v * EPV], 0.0f);
                rv.mask(lane + v * G, &g[u][v * EPV], 0.0f);
            }
        }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const float d = group_reduce<G, OpAdd>(lane_dot<K>(a[u], g[u]));
#pragma unroll
        for (int k = 0; k < K; ++k) a[u][k] = a[u][k] * (g[u][k] - d);
        const int r = r0 + u * step;
        const int64_t o = base + static_cast<int64_t>(r) * cols;
        if constexpr (VEC) {
            const RowVecs<E, SHIFT> rv(o, cols);
#pragma unroll
            for (int v = 0; v < V; ++v) {
                const int vi = lane + v * G;
                if (act[u] && vi < rv.nv) rv.store(dx, vi, &a[u][v * EPV]);
            }
        } else {
#pragma unroll
            for (int k = 0; k < K; ++k) {
                const int j = lane + k * G;
                if (act[u] && j < cols) E::store1(dx + o + j, a[u][k]);
            }
        }
    }
}

// The backward pass in packed tiles (rows of n vectors, n not a power of two, row j of a wave
// on lanes [j n, j n + n)): d = sum(dy * y) by the same tree as the forward pass's reductions,
// then dx = y (dy - d).
template <class E, int U>
__device__ __forceinline__ void rows_packed_bwd(const typename E::T* y, const typename E::T* dy,
                                                typename E::T* dx, int64_t base, int n, int nrows,
                                                int r0, int step, int i, int gb, bool on) {
    constexpr int EPV = E::kEPV;
    const int cols = n * EPV;
    float a[U][EPV], g[U][EPV];
    typename E::R ra[U], rg[U];
    bool act[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t o = base + static_cast<int64_t>(r0 + u * step) * cols + i * EPV;
        act[u] = on && r0 + u * step < nrows;
        ra[u] = act[u] ? E::load_raw(y + o) : E::raw_fill(0.0f);
        rg[u] = act[u] ? E::load_raw(dy + o) : E::raw_fill(0.0f);
    }
    float d[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        E::unpack(ra[u], a[u]);
        E::unpack(rg[u], g[u]);
        d[u] = lane_dot<EPV>(a[u], g[u]);
    }
    seg_reduce<OpAdd, U>(d, i, n, gb);
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
        for (int k = 0; k < EPV; ++k) a[u][k] = a[u][k] * (g[u][k] - d[u]);
        if (act[u])
            E::store_vec(dx + base + static_cast<int64_t>(r0 + u * step) * cols + i * EPV, a[u]);
    }
}

template <class E, int U>
__device__ __forceinline__ uint32_t run_item_packed_bwd(const typename E::T* y,
                                                        const typename E::T* dy,
                                                        typename E::T* dx, int64_t base, int cols,
                                                        int nrows, int reps, int64_t stride,
                                                        int wave, int nwaves, int lane64) {
    const int n = cols / E::kEPV;
    const int rpw = 64 / n;
    const int sub = lane64 / n;
    const int i = lane64 - sub * n;
    const bool on = sub < rpw;
    const int gb = sub * n;
    const int step = nwaves * rpw;
    uint32_t done = 0;
    for (int k = 0; k < reps; ++k) {
        const int64_t b = base + k * stride;
        int r0 = wave * rpw;
        for (; r0 + (U - 1) * step < nrows; r0 += U * step) {
            rows_packed_bwd<E, U>(y, dy, dx, b, n, nrows, r0 + sub, step, i, gb, on);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int left = nrows - (r0 + u * step);
                done += left < rpw ? left : rpw;
            }
        }
        for (; r0 < nrows; r0 += step) {
            rows_packed_bwd<E, 1>(y, dy, dx, b, n, nrows, r0 + sub, step, i, gb, on);
            const int left = nrows - r0;
            done += left < rpw ? left : rpw;
        }
    }
    return done;
}

template <class E, int G, int V, int U, bool VEC, bool SHIFT>
__device__ __forceinline__ uint32_t run_item_bwd(const typename E::T* y, const typename E::T* dy,
                                                 typename E::T* dx, int64_t base, int cols,
                                                 int nrows, int reps, int64_t stride, int wave,
                                                 int nwaves, int lane64) {
    constexpr int RPW = 64 / G;
    const int sub = lane64 / G;
    const int lane = lane64 % G;
    const int step = nwaves * RPW;
    uint32_t done = 0;
    for (int k = 0; k < reps; ++k) {
        const int64_t b = base + k * stride;
        int r0 = wave * RPW;
        // as run_item: U rows per group while the last of them has a row, then one at a time
        for (; r0 + (U - 1) * step < nrows; r0 += U * step) {
            rows_u_bwd<E, G, V, U, VEC, SHIFT>(y, dy, dx, b, cols, nrows, r0 + sub, step, lane);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int left = nrows - (r0 + u * step);
                done += left < RPW ? left : RPW;
            }
        }
        if constexpr (U > 1) {
            for (; r0 < nrows; r0 += step) {
                rows_u_bwd<E, G, V, 1, VEC, SHIFT>(y, dy, dx, b, cols, nrows, r0 + sub, step, lane);
                const int left = nrows - r0;
                done += left < RPW ? left : RPW;
            }
        }
    }
    return done;
}

// One row beyond the tile, one wave: pass 1 streams y and dy once, keeping the lane's partial
// sum of products (each chunk's products by the in-lane tree, chunks in order) and, when both
// fit the wave's LDS region (2 cols <= cap), staging them there; pass 2 forms dx from LDS or,
// otherwise, from a second read of y and dy.  Both variants add in the same order.
template <class E, bool VEC, bool STAGE>
__device__ __forceinline__ void long_row_bwd(const typename E::T* y, const typename E::T* dy,
                                             typename E::T* dx, int cols, int lane, float* lds,
                                             int cap) {
    using L = LongRow<E, VEC, 16>;  // two streams: half the values per lane per chunk
    constexpr int K = L::K;
    const int n = L::extent(cols);
    const int step = L::kStep;
    const bool stage = STAGE && 2 * cols <= cap;
    float s = 0.0f;
    for (int first = lane; first < n; first += step) {
        float a[K], g[K];
        L::load(y, cols, first, a, 0.0f);
        L::load(dy, cols, first, g, 0.0f);
        if (stage) {
            L::to_lds(lds, cols, first, a);
            L::to_lds(lds + cols, cols, first, g);
        }
#pragma unroll
        for (int k = 0; k < K; ++k) g[k] *= a[k];
        s += lane_reduce<K, OpAdd>(g);
    }
    const float d = group_reduce<64, OpAdd>(s);
    for (int first = lane; first < n; first += step) {
        float a[K], g[K];
        if (stage) {
            L::from_lds(lds, cols, first, a, 0.0f);
            L::from_lds(lds + cols, cols, first, g, 0.0f);
        } else {
            L::load(y, cols, first, a, 0.0f);
            L::load(dy, cols, first, g, 0.0f);
        }
#pragma unroll
        for (int k = 0; k < K; ++k) a[k] = a[k] * (g[k] - d);
        L::store(dx, cols, first, a);
    }
}

// Backward rows beyond the register tile, one (or two) at a time per workgroup, laid out as
// in team_rows: y and dy held in registers, d = sum dy * y formed by the in-lane tree, the
// wave's butterfly and the waves' values in wave order; one barrier per rows, alternating the
// slot set (`which`), so a set is rewritten only after every wave has passed the next barrier.
template <class E, int L, int U, bool SHIFT>
__device__ __forceinline__ void team_rows_bwd(const typename E::T* y, const typename E::T* dy,
                                              typename E::T* dx, const int64_t (&off)[U],
                                              const bool (&act)[U], int cols, int t, int nt,
                                              int wave, int nwaves, int lane, int which) {
    constexpr int K = L * E::kEPV;
    float a[U][K], g[U][K];
    typename E::R ra[U][L], rg[U][L];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const RowVecs<E, SHIFT> rv(off[u], cols);
        team_load<E, L, SHIFT>(y, rv, t, nt, act[u], ra[u], 0.0f);  // padding: products 0
        team_load<E, L, SHIFT>(dy, rv, t, nt, act[u], rg[u], 0.0f);
    }
    float d[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const RowVecs<E, SHIFT> rv(off[u], cols);
        team_unpack<E, L, SHIFT>(rv, t, nt, ra[u], a[u], 0.0f);
        team_unpack<E, L, SHIFT>(rv, t, nt, rg[u], g[u], 0.0f);
        d[u] = group_reduce<64, OpAdd>(lane_dot<K>(a[u], g[u]));
    }
    team_combine<OpAdd, U>(d, which, wave, nwaves, lane);
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
        for (int k = 0; k < K; ++k) a[u][k] = a[u][k] * (g[u][k] - d[u]);
        team_store<E, L, SHIFT>(dx, RowVecs<E, SHIFT>(off[u], cols), t, nt, act[u], a[u]);
    }
}

// A backward row longer than nt * L vectors: d over chunks, then y and dy read again.
template <class E, int L, bool SHIFT>
__device__ __forceinline__ void team_row_bwd_two_pass(const typename E::T* y,
                                                      const typename E::T* dy, typename E::T* dx,
                                                      int64_t off, int cols, int t, int nt,
                                                      int wave, int nwaves, int lane, int which) {
    constexpr int K = L * E::kEPV;
    const RowVecs<E, SHIFT> rv(off, cols);
    float s = 0.0f;
    for (int first = t; first - t < rv.nv; first += nt * L) {
        float a[K], g[K];
        typename E::R ra[L], rg[L];
        team_load<E, L, SHIFT>(y, rv, first, nt, true, ra, 0.0f);
        team_load<E, L, SHIFT>(dy, rv, first, nt, true, rg, 0.0f);
        team_unpack<E, L, SHIFT>(rv, first, nt, ra, a, 0.0f);
        team_unpack<E, L, SHIFT>(rv, first, nt, rg, g, 0.0f);
#pragma unroll
        for (int k = 0; k < K; ++k) g[k] *= a[k];
        s += lane_reduce<K, OpAdd>(g);
    }
    float d[1] = {group_reduce<64, OpAdd>(s)};
    team_combine<OpAdd, 1>(d, which, wave, nwaves, lane);
    for (int first = t; first - t < rv.nv; first += nt * L) {
        float a[K], g[K];
        typename E::R ra[L], rg[L];
        team_load<E, L, SHIFT>(y, rv, first, nt, true, ra, 0.0f);
        team_load<E, L, SHIFT>(dy, rv, first, nt, true, rg, 0.0f);
        team_unpack<E, L, SHIFT>(rv, first, nt, ra, a, 0.0f);
        team_unpack<E, L, SHIFT>(rv, first, nt, rg, g, 0.0f);
#pragma unroll
        for (int k = 0; k < K; ++k) a[k] = a[k] * (g[k] - d[0]);
        team_store<E, L, SHIFT>(dx, rv, first, nt, true, a);
    }
}

template <class E, int KCLASS, bool SHIFT>
__device__ __forceinline__ uint32_t team_item_bwd(const typename E::T* y, const typename E::T* dy,
                                                  typename E::T* dx, int64_t base, int cols,
                                                  int nrows, int reps, int64_t stride, int wave,
                                                  int nwaves, int lane) {
    const int nt = nwaves * 64;
    const int t = wave * 64 + lane;
    const int per_lane = (span_vecs<E, SHIFT>(cols) + nt - 1) / nt;
    constexpr int kMaxL = kTeamMaxL<E, KCLASS>;  // vectors per lane and stream
    constexpr bool kPair = 2 * 4 * E::kEPV <= bsm::kTeamValues;  // as in team_item
    int which = 0;
    if (kPair && per_lane <= 4) {
        RowWalk<2> w(base, cols, nrows, reps, stride);
        while (w.more()) {
            int64_t off[2];
            bool act[2];
            w.next(off, act);
            team_rows_bwd<E, 4, 2, SHIFT>(y, dy, dx, off, act, cols, t, nt, wave, nwaves, lane,
                                          which);
            which ^= 1;
        }
    } else if (per_lane <= kMaxL) {
        RowWalk<1> w(base, cols, nrows, reps, stride);
        while (w.more()) {
            int64_t off[1];
            bool act[1];
            w.next(off, act);
            team_rows_bwd<E, kMaxL, 1, SHIFT>(y, dy, dx, off, act, cols, t, nt, wave, nwaves,
                                              lane, which);
            which ^= 1;
        }
    } else {
        RowWalk<1> w(base, cols, nrows, reps, stride);
        while (w.more()) {
            int64_t off[1];
            bool act[1];
            w.next(off, act);
            team_row_bwd_two_pass<E, kMaxL, SHIFT>(y, dy, dx, off[0], cols, t, nt, wave, nwaves,
                                                   lane, which);
            which ^= 1;
        }
    }
    // The next item starts again with slot set 0, which this item's last rows may have used:
    // every wave has read its slots before any wave goes on.
    __syncthreads();
    return team_rows_of_wave(nrows, reps, wave, nwaves);
}

// long_row_bwd for a shifted row: the same two passes over the vectors that cover it (outside
// elements read as 0, never written), staged when both streams' vectors fit the wave's LDS
// region.
template <class E, bool STAGE>
__device__ __forceinline__ void long_row_bwd_shift(const typename E::T* y, const typename E::T* dy,
                                                   typename E::T* dx, int64_t o, int cols,
                                                   int lane, float* lds, int cap) {
    constexpr int EPV = E::kEPV;
    constexpr int CH = 16 / EPV;  // vectors per lane and stream per chunk (16 values)
    constexpr int K = CH * EPV;
    const RowVecs<E, true> rv(o, cols);
    const int n = rv.nv;
    const int span = n * EPV;  // floats of one stream staged
    const bool stage = STAGE && 2 * span <= cap;
    float s = 0.0f;
    for (int first = lane; first < n; first += CH * 64) {
        float a[K], g[K];
        typename E::R ra[CH], rg[CH];
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const int vi = first + c * 64;
            ra[c] = vi < n ? E::load_raw(y + rv.start + vi * EPV) : E::raw_fill(0.0f);
            rg[c] = vi < n ? E::load_raw(dy + rv.start + vi * EPV) : E::raw_fill(0.0f);
        }
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const int vi = first + c * 64;
            E::unpack(ra[c], a + c * EPV);
            E::unpack(rg[c], g + c * EPV);
            rv.mask(vi, a + c * EPV, 0.0f);
            rv.mask(vi, g + c * EPV, 0.0f);
            if (stage && vi < n) {
#pragma unroll
                for (int i = 0; i < EPV; i += 4) {
                    *reinterpret_cast<f32x4*>(lds + vi * EPV + i) =
                        f32x4{a[c * EPV + i], a[c * EPV + i + 1], a[c * EPV + i + 2], a[c * EPV + i + 3]};
                    *reinterpret_cast<f32x4*>(lds + span + vi * EPV + i) =
                        f32x4{g[c * EPV + i], g[c * EPV + i + 1], g[c * EPV + i + 2], g[c * EPV + i + 3]};
                }
            }
        }
#pragma unroll
        for (int k = 0; k < K; ++k) g[k] *= a[k];
        s += lane_reduce<K, OpAdd>(g);
    }
    const float d = group_reduce<64, OpAdd>(s);
    for (int first = lane; first < n; first += CH * 64) {
        float a[K], g[K];
        if (stage) {
#pragma unroll
            for (int c = 0; c < CH; ++c) {
                const int vi = first + c * 64;
#pragma unroll
                for (int i = 0; i < EPV; i += 4) {
                    f32x4 va = f32x4{0.0f, 0.0f, 0.0f, 0.0f}, vg = va;
                    if (vi < n) {
                        va = *reinterpret_cast<const f32x4*>(lds + vi * EPV + i);
                        vg = *reinterpret_cast<const f32x4*>(lds + span + vi * EPV + i);
                    }
                    a[c * EPV + i] = va.x; a[c * EPV + i + 1] = va.y;
                    a[c * EPV + i + 2] = va.z; a[c * EPV + i + 3] = va.w;
                    g[c * EPV + i] = vg.x; g[c * EPV + i + 1] = vg.y;
                    g[c * EPV + i + 2] = vg.z; g[c * EPV + i + 3] = vg.w;
                }
            }
        } else {
            typename E::R ra[CH], rg[CH];
#pragma unroll
            for (int c = 0; c < CH; ++c) {
                const int vi = first + c * 64;
                ra[c] = vi < n ? E::load_raw(y + rv.start + vi * EPV) : E::raw_fill(0.0f);
                rg[c] = vi < n ? E::load_raw(dy + rv.start + vi * EPV) : E::raw_fill(0.0f);
            }
#pragma unroll
            for (int c = 0; c < CH; ++c) {
                E::unpack(ra[c], a + c * EPV);
                E::unpack(rg[c], g + c * EPV);
            }
        }
#pragma unroll
        for (int k = 0; k < K; ++k) a[k] = a[k] * (g[k] - d);
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const int vi = first + c * 64;
            if (vi < n) rv.store(dx, vi, a + c * EPV);
        }
    }
}

template <class E, int KCLASS, bool VEC, bool SHIFT>
__device__ __forceinline__ uint32_t dispatch_item_bwd(const typename E::T* y,
                                                      const typename E::T* dy, typename E::T* dx,
                                                      int64_t base, int cols, int nrows, int reps,
                                                      int64_t stride, int wave, int nwaves,
                                                      int lane64, float* lds, int cap, bool team) {
    const int nvec = VEC ? span_vecs<E, SHIFT>(cols) : (cols + E::kEPV - 1) / E::kEPV;
    if constexpr (VEC && KCLASS >= 4) {
        // rows beyond the forward register tile: the workgroup's waves share each row
        if (team && nvec > 512)
            return team_item_bwd<E, KCLASS, SHIFT>(y, dy, dx, base, cols, nrows, reps, stride,
                                                   wave, nwaves, lane64);
    }
#define BSM_RUN_BWD(G, V, U) run_item_bwd<E, G, V, U, VEC, SHIFT>(y, dy, dx, base, cols, nrows, reps, stride, wave, nwaves, lane64)
    if constexpr (VEC) {
        // the tile of bsm::tile_for_bwd (rows of 33..64 vectors keep 64 lanes x 1 vector: with
        // two input streams the forward pass's 32 x 2 tile measured 3% slower on 384 x 512 x
        // 512 bf16)
        constexpr bool F = E::kBytes == 4;
        const bsm::Tile t = bsm::tile_for_bwd(nvec, KCLASS < 3 ? KCLASS : 3, E::kBytes, !SHIFT);
        if constexpr (!SHIFT && KCLASS == 0) {
            if ((t.G & (t.G - 1)) != 0)  // packed tile
                return run_item_packed_bwd<E, 2>(y, dy, dx, base, cols, nrows, reps, stride, wave,
                                                 nwaves, lane64);
        }
#define BSM_TILE(g, v, u) if (t.G == g && t.V == v && t.U == u) return BSM_RUN_BWD(g, v, u)
        if constexpr (KCLASS == 0) BSM_TILE(8, 1, 2);
        BSM_TILE(16, 1, 2);
        if constexpr (F) BSM_TILE(32, 1, 4);
        BSM_TILE(32, 1, 2);
        if constexpr (KCLASS >= 1) {
            if constexpr (F) {
                BSM_TILE(64, 1, 4);
                BSM_TILE(64, 2, 2);
            }
            BSM_TILE(64, 1, 2);
            BSM_TILE(64, 2, 1);
        }
        if constexpr (KCLASS >= 2) BSM_TILE(64, 4, 1);
        if constexpr (F && KCLASS >= 3) BSM_TILE(64, 8, 1);
#undef BSM_TILE
    } else {
        if (nvec <= 16) return BSM_RUN_BWD(16, 1, 1);
        if (nvec <= 32) return BSM_RUN_BWD(32, 1, 1);
        if (nvec <= 64) return BSM_RUN_BWD(64, 1, 1);
    }
#undef BSM_RUN_BWD
    if constexpr (!VEC || KCLASS >= 3) {
        uint32_t done = 0;
        for (int k = 0; k < reps; ++k) {
            for (int r = wave; r < nrows; r += nwaves) {
                const int64_t o = base + k * stride + static_cast<int64_t>(r) * cols;
                if constexpr (VEC && SHIFT)
                    long_row_bwd_shift<E, (KCLASS >= 4)>(y, dy, dx, o, cols, lane64, lds, cap);
                else
                    long_row_bwd<E, VEC, (KCLASS >= 4)>(y + o, dy + o, dx + o, cols, lane64, lds,
                                                        cap);
                ++done;
            }
        }
        return done;
    }
    return 0;  // unreachable: the item's access path is chosen so that its class covers it
}

// Worker w of the table is workgroup w (all its waves share each item) or, when per_wave is
// set, wave (w * waves_per_workgroup + wave), which then runs its own items alone.  BWD selects
// the backward op (a = y, b = dy, out = dx); the forward op reads a only.
template <class E, int KCLASS, bool BWD, bool SHIFTED>
__device__ __forceinline__ void worker_loop(const typename E::T* a, const typename E::T* b,
                                            typename E::T* out, const int32_t* __restrict__ worker_ptr,
                                            const bsm_item* __restrict__ items, int base_aligned,
                                            int per_wave, int lds_floats_per_wave,
                                            bsm_trace_rec* __restrict__ trace, float* lds_base) {
    const int w = blockIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
    const int nwaves = static_cast<int>(blockDim.x) >> 6;
    const int lane64 = static_cast<int>(threadIdx.x) & 63;
    const uint64_t t0 = trace ? __builtin_amdgcn_s_memrealtime() : 0;
    const int worker = per_wave ? w * nwaves + wave : w;
    const int my_wave = per_wave ? 0 : wave;
    const int my_nwaves = per_wave ? 1 : nwaves;
    float* const lds = lds_base + wave * lds_floats_per_wave;
    uint32_t rows = 0;
    const int i0 = worker_ptr[worker];
    const int i1 = worker_ptr[worker + 1];
    for (int i = i0; i < i1; ++i) {
        const int64_t base = items[i].elem_offset;
        const int cols = items[i].cols;
        const int nrows = items[i].nrows;
        const int reps = items[i].reps;
        const int64_t stride = static_cast<int64_t>(items[i].rep_stride) * cols;
        // Access path: whole 16-byte vectors when every row of the item starts and ends on
        // one; shifted vectors when the buffers are aligned but the rows are not (in the
        // instances for plans with such slices, SHIFTED, and as long as the kernel class has a
        // tile or path for the extra vector); else element by element.
        const bool rows_whole = ((base | static_cast<int64_t>(cols)) & (E::kEPV - 1)) == 0;
        const int span = span_vecs<E, true>(cols);
        const bool shift_fits = SHIFTED && (BWD ? (KCLASS >= 3 || span <= kClassMaxVecs<KCLASS>)
                                                : span <= kClassMaxVecs<KCLASS>);
        const int path = !base_aligned ? 0 : rows_whole ? 1 : shift_fits ? 2 : 0;
#define BSM_ARGS_TAIL cols, nrows, reps, stride, my_wave, my_nwaves, lane64, lds, lds_floats_per_wave, !per_wave
        if constexpr (BWD) {
            if (path == 1)
                rows += dispatch_item_bwd<E, KCLASS, true, false>(a, b, out, base, BSM_ARGS_TAIL);
            else if (SHIFTED && path == 2)
                rows += dispatch_item_bwd<E, KCLASS, true, SHIFTED>(a, b, out, base, BSM_ARGS_TAIL);
            else
                rows += dispatch_item_bwd<E, KCLASS, false, false>(a, b, out, base, BSM_ARGS_TAIL);
        } else {
            if (path == 1)
                rows += dispatch_item<E, KCLASS, true, false>(a, out, base, BSM_ARGS_TAIL);
            else if (SHIFTED && path == 2)
                rows += dispatch_item<E, KCLASS, true, SHIFTED>(a, out, base, BSM_ARGS_TAIL);
            else
                rows += dispatch_item<E, KCLASS, false, false>(a, out, base, BSM_ARGS_TAIL);
        }
#undef BSM_ARGS_TAIL
    }
    if (trace && lane64 == 0) {
        bsm_trace_rec rec;
        rec.wg = static_cast<uint32_t>(w);
        // XCC_ID register (id 20), bits [3:0]; HW_ID register (id 4), all 32 bits
        rec.xcc_id = __builtin_amdgcn_s_getreg(20 | (0 << 6) | ((4 - 1) << 11)) & 0xF;
        rec.hw_id = __builtin_amdgcn_s_getreg(4 | (0 << 6) | ((32 - 1) << 11));
        rec.rows = rows;
        rec.t_start = t0;
        rec.t_end = __builtin_amdgcn_s_memrealtime();
        trace[static_cast<int64_t>(w) * nwaves + wave] = rec;
    }
}

extern __shared__ float bsm_lds[];  // lds_floats_per_wave floats per wave (long rows only)

// Launch bounds: any workgroup size up to 1024 threads (128 VGPRs per lane); long-row plans run
// workgroups of bsm::team_threads(class) threads (classes 4 and 5: 256, two or more per CU;
// class 6: 512, one per CU), so their rows may hold up to 256 VGPRs per lane.  bf16 plans of
// class 3 run workgroups of at most 256 threads: their 64 x 8 tile needs about 160 VGPRs (at
// 128 it spilled, 4.7-4.8 TB/s on 2304-4096-element rows; at 163 it runs three waves per SIMD,
// 5.0-5.2 TB/s).
template <class E, int KCLASS>
constexpr int kMaxThreads = KCLASS >= 4 ? bsm::team_threads(KCLASS)
                                        : (E::kBytes == 2 && KCLASS == 3 ? 256 : 1024);
template <class E, int KCLASS>
constexpr int kMinWavesPerSimd = (KCLASS >= 4 || (E::kBytes == 2 && KCLASS == 3)) ? 2 : 1;

// SHIFTED: the instance for plans with slices whose rows do not start and end on 16-byte
// vectors (kept apart so that the other plans' instances carry none of its registers).
template <class E, int KCLASS, bool SHIFTED>
__global__ void __launch_bounds__((kMaxThreads<E, KCLASS>), (kMinWavesPerSimd<E, KCLASS>))
bsm_softmax_kernel(const typename E::T* in, typename E::T* out, const int32_t* __restrict__ worker_ptr,
                   const bsm_item* __restrict__ items, int base_aligned, int per_wave,
                   int lds_floats_per_wave, bsm_trace_rec* __restrict__ trace) {
    worker_loop<E, KCLASS, false, SHIFTED>(in, nullptr, out, worker_ptr, items, base_aligned,
                                           per_wave, lds_floats_per_wave, trace, bsm_lds);
}

// dx = softmax backward of (y, dy) under the same work table.
template <class E, int KCLASS, bool SHIFTED>
__global__ void __launch_bounds__((kMaxThreads<E, KCLASS>), (kMinWavesPerSimd<E, KCLASS>))
bsm_softmax_bwd_kernel(const typename E::T* y, const typename E::T* dy, typename E::T* dx,
                       const int32_t* __restrict__ worker_ptr, const bsm_item* __restrict__ items,
                       int base_aligned, int per_wave, int lds_floats_per_wave,
                       bsm_trace_rec* __restrict__ trace) {
    worker_loop<E, KCLASS, true, SHIFTED>(y, dy, dx, worker_ptr, items, base_aligned, per_wave,
                                          lds_floats_per_wave, trace, bsm_lds);
}

}  // namespace bsm_dev
