// Host launch wrappers of the persistent softmax kernels (device code in bsm_device.hpp,
// instances in bsm_kernels_*.hip) and the streaming copy kernel, defined here.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "bsm.h"
#include "bsm_device.hpp"
#include "bsm_kernel_set.hpp"
#include "bsm_launch.hpp"

namespace {

using namespace bsm_dev;

// Streaming copy, the bandwidth reference: nontemporal 16-byte accesses, grid-stride, so the
// whole grid sweeps one compact window (the fastest copy layout measured on MI355X); a byte
// loop handles an unaligned remainder.
__global__ void __launch_bounds__(256) bsm_copy_kernel(const u32x4* __restrict__ src,
                                                       u32x4* __restrict__ dst, int64_t n_vec) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * 256;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < n_vec; i += stride)
        __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

__global__ void __launch_bounds__(256) bsm_copy_bytes_kernel(const unsigned char* __restrict__ src,
                                                             unsigned char* __restrict__ dst,
                                                             int64_t n) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * 256;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < n; i += stride)
        dst[i] = src[i];
}

// Both ops take (a, [b,] out, worker_ptr, items, aligned, per_wave, lds_floats, trace); the
// forward op has no b.
hipError_t launch_fn(const void* fn, bool bwd, const void* a, const void* b, void* out,
                     const int32_t* worker_ptr, const bsm_item* items, int n_wg, int wg_threads,
                     int aligned, int per_wave, int lds_floats, void* trace, hipStream_t stream) {
    const size_t lds_bytes = static_cast<size_t>(lds_floats) * sizeof(float) * (wg_threads / 64);
    void* args_fwd[] = {&a, &out, &worker_ptr, &items, &aligned, &per_wave, &lds_floats, &trace};
    void* args_bwd[] = {&a, &b, &out, &worker_ptr, &items, &aligned, &per_wave, &lds_floats, &trace};
    // hipLaunchKernel reports a failed launch itself, without touching the thread's last error
    return hipLaunchKernel(fn, dim3(n_wg), dim3(wg_threads), bwd ? args_bwd : args_fwd, lds_bytes,
                           stream);
}

// The instances live in four sources (element type x access set) that compile in parallel.
const void* fn_for(bsm_dtype dtype, bool temporal, int kclass, bool shifted, bool bwd) {
    if (dtype == BSM_BF16)
        return shifted ? bsm::softmax_fn_bf16_shifted(kclass, temporal, bwd)
                       : bsm::softmax_fn_bf16(kclass, temporal, bwd);
    return shifted ? bsm::softmax_fn_f32_shifted(kclass, temporal, bwd)
                   : bsm::softmax_fn_f32(kclass, temporal, bwd);
}

}  // namespace

namespace bsm {

int kernel_class_for(int32_t max_cols, int elem_bytes, bool shifted) {
    const int64_t nvec = (static_cast<int64_t>(max_cols) * elem_bytes + kVecBytes - 1) / kVecBytes +
                         (shifted ? 1 : 0);
    if (nvec <= 32) return 0;
    if (nvec <= 128) return 1;  // rows of 33..64 vectors run 32 lanes x 2 vectors
    if (nvec <= 256) return 2;
    if (nvec <= 512) return 3;
    // longer rows: workgroup-held, up to kTeamValues values per lane in class 4
    const int64_t elems = nvec * (kVecBytes / elem_bytes);
    if (elems <= kTeamThreads * kTeamValues) return 4;
    return elems <= 2 * kTeamThreads * kTeamValues ? 5 : kLongestClass;
}

hipError_t launch_softmax(bsm_dtype dtype, int kernel_class, bool shifted, bool temporal,
                          const void* in, void* out, const int32_t* d_worker_ptr,
                          const bsm_item* d_items, int n_wg, int wg_threads, int per_wave,
                          int lds_floats_per_wave, void* trace, hipStream_t stream) {
    const int aligned = ((reinterpret_cast<uintptr_t>(in) | reinterpret_cast<uintptr_t>(out)) & 15) == 0;
    return launch_fn(fn_for(dtype, temporal, kernel_class, shifted, false), false, in, nullptr, out,
                     d_worker_ptr, d_items, n_wg, wg_threads, aligned, per_wave,
                     lds_floats_per_wave, trace, stream);
}

hipError_t launch_softmax_backward(bsm_dtype dtype, int kernel_class, bool shifted, bool temporal,
                                   const void* y, const void* dy, void* dx,
                                   const int32_t* d_worker_ptr, const bsm_item* d_items, int n_wg,
                                   int wg_threads, int per_wave, int lds_floats_per_wave,
                                   void* trace, hipStream_t stream) {
    const int aligned = ((reinterpret_cast<uintptr_t>(y) | reinterpret_cast<uintptr_t>(dy) |
                          reinterpret_cast<uintptr_t>(dx)) & 15) == 0;
    return launch_fn(fn_for(dtype, temporal, kernel_class, shifted, true), true, y, dy, dx,
                     d_worker_ptr, d_items, n_wg, wg_threads, aligned, per_wave,
                     lds_floats_per_wave, trace, stream);
}

// Largest static LDS of the plan's instances (forward and backward, both cache policies).
hipError_t static_lds_bytes(bsm_dtype dtype, int kernel_class, bool shifted, int* bytes) {
    *bytes = 0;
    for (int temporal = 0; temporal < 2; ++temporal)
        for (int bwd = 0; bwd < 2; ++bwd) {
            hipFuncAttributes a;
            const hipError_t e =
                hipFuncGetAttributes(&a, fn_for(dtype, temporal != 0, kernel_class, shifted, bwd != 0));
            if (e != hipSuccess) return e;
            if (static_cast<int>(a.sharedSizeBytes) > *bytes) *bytes = static_cast<int>(a.sharedSizeBytes);
        }
    return hipSuccess;
}

// Resident workgroups per CU of the plan's forward instance.
hipError_t resident_wgs_per_cu(bsm_dtype dtype, int kernel_class, bool shifted, int wg_threads,
                               size_t dyn_lds_bytes, int* n) {
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(
        n, fn_for(dtype, false, kernel_class, shifted, false), wg_threads, dyn_lds_bytes);
}

hipError_t launch_copy(const void* src, void* dst, int64_t bytes, int n_cu, hipStream_t stream) {
    const bool aligned = ((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) & 15) == 0;
    const int64_t n_vec = aligned ? bytes / 16 : 0;
    const int64_t max_grid = static_cast<int64_t>(n_cu > 0 ? n_cu : 256) * 4;
    if (n_vec > 0) {
        int64_t grid = (n_vec + 255) / 256;
        if (grid > max_grid) grid = max_grid;
        const u32x4* a_src = static_cast<const u32x4*>(src);
        u32x4* a_dst = static_cast<u32x4*>(dst);
        int64_t a_n = n_vec;
        void* args[] = {&a_src, &a_dst, &a_n};
        const hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(&bsm_copy_kernel),
                                             dim3(static_cast<unsigned>(grid)), dim3(256), args, 0,
                                             stream);
        if (e != hipSuccess) return e;
    }
    const int64_t rest = bytes - n_vec * 16;
    if (rest > 0) {
        int64_t grid = (rest + 255) / 256;
        if (grid > max_grid) grid = max_grid;
        const unsigned char* a_src = static_cast<const unsigned char*>(src) + n_vec * 16;
        unsigned char* a_dst = static_cast<unsigned char*>(dst) + n_vec * 16;
        int64_t a_n = rest;
        void* args[] = {&a_src, &a_dst, &a_n};
        return hipLaunchKernel(reinterpret_cast<const void*>(&bsm_copy_bytes_kernel),
                               dim3(static_cast<unsigned>(grid)), dim3(256), args, 0, stream);
    }
    return hipSuccess;
}

}  // namespace bsm
