// Host launch wrappers of the batched matrix-product kernels (device code in bsm_gemm.hpp).
#include <hip/hip_runtime.h>

#include <cstdint>

#include "bsm.h"
#include "bsm_gemm.hpp"
#include "bsm_launch.hpp"

namespace {

using bsm_mm::Shape;

template <int MODE, bool BF16OUT, bool VEC, bool TEMPORAL, bool AREG>
hipError_t launch_g(const void* a, const void* b, void* c, const Shape& s, const int32_t* worker_ptr,
                    const bsm_item* items, int n_wg, void* trace, hipStream_t stream) {
    const uint16_t* a_a = static_cast<const uint16_t*>(a);
    const uint16_t* a_b = static_cast<const uint16_t*>(b);
    void* a_c = c;
    Shape a_s = s;
    bsm_trace_rec* a_trace = static_cast<bsm_trace_rec*>(trace);
    void* args[] = {&a_a, &a_b, &a_c, &a_s, &worker_ptr, &items, &a_trace};
    // single-pass instances: the last flag selects the deep form (64 < k <= 128)
    const size_t lds = static_cast<size_t>(MODE == bsm_mm::kModeNtSoftmax1 ? bsm_mm::s1_lds_bytes(BF16OUT, AREG)
                                                                         : bsm_mm::wg_lds_bytes(BF16OUT));
    return hipLaunchKernel(reinterpret_cast<const void*>(&bsm_mm::bsm_gemm_kernel<MODE, BF16OUT, VEC, TEMPORAL, AREG>),
                           dim3(n_wg), dim3(bsm_mm::kGemmThreads), args, lds, stream);
}

}  // namespace

namespace bsm {

int gemm_wg_threads() { return bsm_mm::kGemmThreads; }
bool gemm_single_pass_shape(int n, int k) { return bsm_mm::single_pass_shape(n, k); }
int gemm_lds_bytes_per_wg(bool bf16_out, bool single_pass) {
    return single_pass ? bsm_mm::s1_lds_bytes(bf16_out, true) : bsm_mm::wg_lds_bytes(bf16_out);
}
int gemm_waves_per_simd(bool single_pass) {
    return single_pass ? bsm_mm::kS1WavesPerSimd : bsm_mm::kWavesPerSimd;
}
int gemm_rows_per_wg(bool single_pass) {
    return single_pass ? bsm_mm::kS1Rows : bsm_mm::kWaves * bsm_mm::kTileM;
}

hipError_t launch_gemm(int layout, bool bf16_out, bool temporal, bool single_pass, const void* a,
                       const void* b, void* c, int m, int n, int k, float alpha,
                       const int32_t* d_worker_ptr, const bsm_item* d_items, int n_wg, void* trace,
                       hipStream_t stream) {
    Shape s;
    s.m = m;
    s.n = n;
    s.k = k;
    s.a_batch = static_cast<int64_t>(m) * k;
    s.b_batch = static_cast<int64_t>(n) * k;
    s.c_batch = static_cast<int64_t>(m) * n;
    s.alpha = alpha;
    // 16-byte operand pieces and 16-byte output stores (4 fp32 or 8 bf16 columns): rows of A
    // (and NT's B) of k elements, rows of NN's B and of C of n elements, every base 16-byte
    // aligned
    const uintptr_t ptrs = reinterpret_cast<uintptr_t>(a) | reinterpret_cast<uintptr_t>(b) |
                           reinterpret_cast<uintptr_t>(c);
    const bool vec = (ptrs & 15) == 0 && k % 8 == 0 &&
                     n % ((layout == bsm_mm::kNN || bf16_out) ? 8 : 4) == 0;
    const bool areg = bsm_mm::use_areg(vec, n, k);
#define BSM_G(M, O, V, T, R) launch_g<M, O, V, T, R>(a, b, c, s, d_worker_ptr, d_items, n_wg, trace, stream)
#define BSM_GV(M, O, T) (!vec ? BSM_G(M, O, false, T, false) \
                              : (areg ? BSM_G(M, O, true, T, true) : BSM_G(M, O, true, T, false)))
#define BSM_G1(M, T) (bf16_out ? BSM_GV(M, true, T) : BSM_GV(M, false, T))
#define BSM_G2(M) (temporal ? BSM_G1(M, true) : BSM_G1(M, false))
    // the one-pass softmax takes alpha != 0 only (with alpha = 0 every logit is 0, which the
    // two-pass form handles)
    if (layout == bsm_mm::kModeNtSoftmax && single_pass && vec && alpha != 0.0f &&
        bsm_mm::single_pass_shape(n, k)) {
        // the last flag of the single-pass instance: 64 < k <= 128 (A kept in LDS)
#define BSM_G1P(O, T) (k > bsm_mm::kChunkK ? BSM_G(bsm_mm::kModeNtSoftmax1, O, true, T, true) \
                                           : BSM_G(bsm_mm::kModeNtSoftmax1, O, true, T, false))
        if (bf16_out) return temporal ? BSM_G1P(true, true) : BSM_G1P(true, false);
        return temporal ? BSM_G1P(false, true) : BSM_G1P(false, false);
#undef BSM_G1P
    }
    if (layout == bsm_mm::kNN) return BSM_G2(bsm_mm::kModeNn);
    if (layout == bsm_mm::kModeNtSoftmax) return BSM_G2(bsm_mm::kModeNtSoftmax);
    return BSM_G2(bsm_mm::kModeNt);
#undef BSM_G2
#undef BSM_G1
#undef BSM_GV
#undef BSM_G
}

}  // namespace bsm
