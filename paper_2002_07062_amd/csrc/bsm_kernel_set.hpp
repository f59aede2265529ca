// The softmax kernel instances of one element type and access set (aligned or shifted rows):
// forward and backward, every kernel class, both cache policies.  Each of the four
// bsm_kernels_<type>[_shifted].hip sources instantiates one set.
#pragma once

#include "bsm_device.hpp"

namespace bsm {

template <class E, bool SHIFTED>
const void* softmax_fn(int kclass, bool bwd) {
#define BSM_FN(K)                                                                                   \
    return bwd ? reinterpret_cast<const void*>(&bsm_dev::bsm_softmax_bwd_kernel<E, K, SHIFTED>)     \
               : reinterpret_cast<const void*>(&bsm_dev::bsm_softmax_kernel<E, K, SHIFTED>)
    switch (kclass) {
        case 0: BSM_FN(0);
        case 1: BSM_FN(1);
        case 2: BSM_FN(2);
        case 3: BSM_FN(3);
        case 4: BSM_FN(4);
        case 5: BSM_FN(5);
        default: BSM_FN(6);
    }
#undef BSM_FN
}

// temporal: ordinary (cache-resident) accesses; otherwise nontemporal.
template <template <bool> class E, bool SHIFTED>
const void* kernel_set(int kclass, bool temporal, bool bwd) {
    return temporal ? softmax_fn<E<false>, SHIFTED>(kclass, bwd)
                    : softmax_fn<E<true>, SHIFTED>(kclass, bwd);
}

const void* softmax_fn_f32(int kclass, bool temporal, bool bwd);
const void* softmax_fn_f32_shifted(int kclass, bool temporal, bool bwd);
const void* softmax_fn_bf16(int kclass, bool temporal, bool bwd);
const void* softmax_fn_bf16_shifted(int kclass, bool temporal, bool bwd);

}  // namespace bsm
