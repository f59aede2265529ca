// Softmax kernel instances, fp32, for plans with rows that do not start or end on 16-byte
// vectors (read as shifted vectors).
#include <hip/hip_runtime.h>

#include "bsm_kernel_set.hpp"

namespace bsm {

const void* softmax_fn_f32_shifted(int kclass, bool temporal, bool bwd) {
    return kernel_set<bsm_dev::F32, true>(kclass, temporal, bwd);
}

}  // namespace bsm
