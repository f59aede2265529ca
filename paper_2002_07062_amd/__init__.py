"""Batched row softmax with slice-to-workgroup scheduling for AMD Instinct MI355X (gfx950).

The product is libbsm.so (C ABI in include/bsm.h: HIP kernels, host planner, plan cache);
this package is its ctypes binding. Build with `python -m paper_2002_07062_amd.build`.
"""

from .bsm import (  # noqa: F401
    BSM_BF16, BSM_ERR_ALIAS, BSM_ERR_HIP, BSM_ERR_INVALID_ARG, BSM_ERR_OOM, BSM_ERR_UNSUPPORTED,
    BSM_F32, BSM_FLAG_CONTIGUOUS_BANKS, BSM_NOALLOC_SCRATCH_BYTES, BSM_FLAG_TEMPORAL, BSM_OK, BSM_SCHED_BALANCED, BSM_SCHED_RR, BSM_SCHED_XCD, DTYPES, ITEM_DTYPE,
    LIB_PATH, SCHEDULES, TRACE_DTYPE, BsmError, Plan, bsm_abi_version, bsm_cache_clear, bsm_copy,
    bsm_default_topology, bsm_device_info, bsm_last_error, bsm_plan_create, bsm_plan_describe,
    bsm_plan_destroy, bsm_plan_execute, bsm_plan_execute_backward, bsm_plan_export, bsm_softmax,
    bsm_softmax_backward, bsm_softmax_noalloc, bsm_status_string, BSM_GEMM_NN, BSM_GEMM_NT, BSM_GEMM_NT_SOFTMAX,
    GEMM_LAYOUTS, bsm_gemm,
    bsm_gemm_execute, bsm_gemm_plan_create,
    bsm_topology, load)
