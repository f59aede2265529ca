// Softmax kernel instances, bf16, for plans whose rows all start and end on 16-byte vectors
// (and for any plan on buffers that are not 16-byte aligned).
#include <hip/hip_runtime.h>

#include "bsm_kernel_set.hpp"

namespace bsm {

const void* softmax_fn_bf16(int kclass, bool temporal, bool bwd) {
    return kernel_set<bsm_dev::BF16, false>(kclass, temporal, bwd);
}

}  // namespace bsm
