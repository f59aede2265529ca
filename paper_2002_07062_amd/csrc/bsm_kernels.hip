// Host launch wrappers of the persistent softmax and copy kernels (device code in
// bsm_device.hpp).
#include <hip/hip_runtime.h>

#include <cstdint>

#include "bsm.h"
#include "bsm_device.hpp"
#include "bsm_launch.hpp"

namespace {

using namespace bsm_dev;

template <class E, int KCLASS>
hipError_t launch_t(const void* in, void* out, const int32_t* worker_ptr, const bsm_item* items,
                    int n_wg, int wg_threads, int aligned, int per_wave, int lds_floats,
                    void* trace, hipStream_t stream) {
    const size_t lds_bytes = static_cast<size_t>(lds_floats) * sizeof(float) * (wg_threads / 64);
    const typename E::T* a_in = static_cast<const typename E::T*>(in);
    typename E::T* a_out = static_cast<typename E::T*>(out);
    bsm_trace_rec* a_trace = static_cast<bsm_trace_rec*>(trace);
    void* args[] = {&a_in, &a_out, &worker_ptr, &items, &aligned, &per_wave, &lds_floats, &a_trace};
    // hipLaunchKernel reports a failed launch itself, without touching the thread's last error
    return hipLaunchKernel(reinterpret_cast<const void*>(&bsm_softmax_kernel<E, KCLASS>),
                           dim3(n_wg), dim3(wg_threads), args, lds_bytes, stream);
}

template <class E>
hipError_t launch_class(int kclass, const void* in, void* out, const int32_t* worker_ptr,
                        const bsm_item* items, int n_wg, int wg_threads, int aligned, int per_wave,
                        int lds_floats, void* trace, hipStream_t stream) {
#define BSM_LAUNCH(K) launch_t<E, K>(in, out, worker_ptr, items, n_wg, wg_threads, aligned, per_wave, lds_floats, trace, stream)
    switch (kclass) {
        case 0: return BSM_LAUNCH(0);
        case 1: return BSM_LAUNCH(1);
        case 2: return BSM_LAUNCH(2);
        case 3: return BSM_LAUNCH(3);
        case 4: return BSM_LAUNCH(4);
        default: return BSM_LAUNCH(5);
    }
#undef BSM_LAUNCH
}

template <class E, int KCLASS>
hipError_t launch_bwd_t(const void* y, const void* dy, void* dx, const int32_t* worker_ptr,
                        const bsm_item* items, int n_wg, int wg_threads, int aligned, int per_wave,
                        int lds_floats, void* trace, hipStream_t stream) {
    const size_t lds_bytes = static_cast<size_t>(lds_floats) * sizeof(float) * (wg_threads / 64);
    const typename E::T* a_y = static_cast<const typename E::T*>(y);
    const typename E::T* a_dy = static_cast<const typename E::T*>(dy);
    typename E::T* a_dx = static_cast<typename E::T*>(dx);
    bsm_trace_rec* a_trace = static_cast<bsm_trace_rec*>(trace);
    void* args[] = {&a_y, &a_dy, &a_dx, &worker_ptr, &items, &aligned, &per_wave, &lds_floats, &a_trace};
    return hipLaunchKernel(reinterpret_cast<const void*>(&bsm_softmax_bwd_kernel<E, KCLASS>),
                           dim3(n_wg), dim3(wg_threads), args, lds_bytes, stream);
}

template <class E>
hipError_t launch_class_bwd(int kclass, const void* y, const void* dy, void* dx,
                            const int32_t* worker_ptr, const bsm_item* items, int n_wg,
                            int wg_threads, int aligned, int per_wave, int lds_floats, void* trace,
                            hipStream_t stream) {
#define BSM_LAUNCH(K) launch_bwd_t<E, K>(y, dy, dx, worker_ptr, items, n_wg, wg_threads, aligned, per_wave, lds_floats, trace, stream)
    switch (kclass) {
        case 0: return BSM_LAUNCH(0);
        case 1: return BSM_LAUNCH(1);
        case 2: return BSM_LAUNCH(2);
        case 3: return BSM_LAUNCH(3);
        case 4: return BSM_LAUNCH(4);
        default: return BSM_LAUNCH(5);
    }
#undef BSM_LAUNCH
}

}  // namespace

namespace bsm {

int kernel_class_for(int32_t max_cols, int elem_bytes) {
    const int64_t nvec = (static_cast<int64_t>(max_cols) * elem_bytes + kVecBytes - 1) / kVecBytes;
    if (nvec <= 32) return 0;
    if (nvec <= 128) return 1;  // rows of 33..64 vectors run 32 lanes x 2 vectors
    if (nvec <= 256) return 2;
    if (nvec <= 512) return 3;
    // longer rows: workgroup-held, up to kTeamValues values per lane in class 4
    return max_cols <= kTeamThreads * kTeamValues ? 4 : 5;
}

hipError_t launch_softmax(bsm_dtype dtype, int kernel_class, bool temporal, const void* in,
                          void* out, const int32_t* d_worker_ptr, const bsm_item* d_items,
                          int n_wg, int wg_threads, int per_wave, int lds_floats_per_wave,
                          void* trace, hipStream_t stream) {
    const int aligned = ((reinterpret_cast<uintptr_t>(in) | reinterpret_cast<uintptr_t>(out)) & 15) == 0;
#define BSM_ARGS kernel_class, in, out, d_worker_ptr, d_items, n_wg, wg_threads, aligned, per_wave, lds_floats_per_wave, trace, stream
    if (dtype == BSM_BF16)
        return temporal ? launch_class<BF16<false>>(BSM_ARGS) : launch_class<BF16<true>>(BSM_ARGS);
    return temporal ? launch_class<F32<false>>(BSM_ARGS) : launch_class<F32<true>>(BSM_ARGS);
#undef BSM_ARGS
}

hipError_t launch_softmax_backward(bsm_dtype dtype, int kernel_class, bool temporal, const void* y,
                                   const void* dy, void* dx, const int32_t* d_worker_ptr,
                                   const bsm_item* d_items, int n_wg, int wg_threads, int per_wave,
                                   int lds_floats_per_wave, void* trace, hipStream_t stream) {
    const int aligned = ((reinterpret_cast<uintptr_t>(y) | reinterpret_cast<uintptr_t>(dy) |
                          reinterpret_cast<uintptr_t>(dx)) & 15) == 0;
#define BSM_ARGS kernel_class, y, dy, dx, d_worker_ptr, d_items, n_wg, wg_threads, aligned, per_wave, lds_floats_per_wave, trace, stream
    if (dtype == BSM_BF16)
        return temporal ? launch_class_bwd<BF16<false>>(BSM_ARGS) : launch_class_bwd<BF16<true>>(BSM_ARGS);
    return temporal ? launch_class_bwd<F32<false>>(BSM_ARGS) : launch_class_bwd<F32<true>>(BSM_ARGS);
#undef BSM_ARGS
}

namespace {
template <class E>
hipError_t static_lds_of(int kernel_class, int* bytes) {
    const void* fns[2] = {nullptr, nullptr};
    switch (kernel_class) {
#define BSM_FNS(K)                                                              \
    case K:                                                                     \
        fns[0] = reinterpret_cast<const void*>(&bsm_softmax_kernel<E, K>);     \
        fns[1] = reinterpret_cast<const void*>(&bsm_softmax_bwd_kernel<E, K>); \
        break;
        BSM_FNS(0)
        BSM_FNS(1)
        BSM_FNS(2)
        BSM_FNS(3)
        BSM_FNS(4)
        default:
            fns[0] = reinterpret_cast<const void*>(&bsm_softmax_kernel<E, 5>);
            fns[1] = reinterpret_cast<const void*>(&bsm_softmax_bwd_kernel<E, 5>);
            break;
#undef BSM_FNS
    }
    *bytes = 0;
    for (const void* fn : fns) {
        hipFuncAttributes a;
        const hipError_t e = hipFuncGetAttributes(&a, fn);
        if (e != hipSuccess) return e;
        if (static_cast<int>(a.sharedSizeBytes) > *bytes) *bytes = static_cast<int>(a.sharedSizeBytes);
    }
    return hipSuccess;
}
}  // namespace

// Static LDS is the same for the streaming and the cache-resident instances; both are checked
// anyway, as they are separate functions.
hipError_t static_lds_bytes(bsm_dtype dtype, int kernel_class, int* bytes) {
    int a = 0, b = 0;
    hipError_t e = dtype == BSM_BF16 ? static_lds_of<BF16<true>>(kernel_class, &a)
                                     : static_lds_of<F32<true>>(kernel_class, &a);
    if (e == hipSuccess)
        e = dtype == BSM_BF16 ? static_lds_of<BF16<false>>(kernel_class, &b)
                              : static_lds_of<F32<false>>(kernel_class, &b);
    *bytes = a > b ? a : b;
    return e;
}

hipError_t resident_wgs_per_cu(bsm_dtype dtype, int kernel_class, int wg_threads,
                               size_t dyn_lds_bytes, int* n) {
    const void* fn = nullptr;
    if (dtype == BSM_BF16) {
        switch (kernel_class) {
            case 0: fn = reinterpret_cast<const void*>(&bsm_softmax_kernel<BF16<true>, 0>); break;
            case 1: fn = reinterpret_cast<const void*>(&bsm_softmax_kernel<BF16<true>, 1>); break;
            case 2: fn = reinterpret_cast<const void*>(&bsm_softmax_kernel<BF16<true>, 2>); break;
            case 3: fn = reinterpret_cast<const void*>(&bsm_softmax_kernel<BF16<true>, 3>); break;
            case 4: fn = reinterpret_cast<const void*>(&bsm_softmax_kernel<BF16<true>, 4>); break;
            default: fn = reinterpret_cast<const void*>(&bsm_softmax_kernel<BF16<true>, 5>); break;
        }
    } else {
        switch (kernel_class) {
            case 0: fn = reinterpret_cast<const void*>(&bsm_softmax_kernel<F32<true>, 0>); break;
            case 1: fn = reinterpret_cast<const void*>(&bsm_softmax_kernel<F32<true>, 1>); break;
            case 2: fn = reinterpret_cast<const void*>(&bsm_softmax_kernel<F32<true>, 2>); break;
            case 3: fn = reinterpret_cast<const void*>(&bsm_softmax_kernel<F32<true>, 3>); break;
            case 4: fn = reinterpret_cast<const void*>(&bsm_softmax_kernel<F32<true>, 4>); break;
            default: fn = reinterpret_cast<const void*>(&bsm_softmax_kernel<F32<true>, 5>); break;
        }
    }
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(n, fn, wg_threads, dyn_lds_bytes);
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
