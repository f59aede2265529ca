// Launch wrappers exported by bsm_kernels.hip to the C-ABI layer (internal).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "bsm.h"

namespace bsm {

// Kernel classes: the longest row decides how large a register tile the kernel instance
// carries (a bigger tile costs registers, hence occupancy, for every row).
//   0: rows of <= 32 16-byte vectors   (fp32 C <= 128,  bf16 C <= 256; tiles up to 64)
//   1: <= 128 vectors                  (fp32 C <= 512,  bf16 C <= 1024)
//   2: <= 256 vectors                  (fp32 C <= 1024, bf16 C <= 2048)
//   3: <= 512 vectors                  (fp32 C <= 2048, bf16 C <= 4096)
//   4: <= 8192 elements, held by a 256-thread workgroup (up to 32 values per lane)
//   5: <= 16384 elements, held by a 256-thread workgroup (up to 64 values per lane)
//   6: any length (a 512-thread workgroup holds up to 32768 elements, longer rows read twice)
// Kernel instance for a plan whose longest row is max_cols elements; `shifted`: some slice's
// rows do not start and end on 16-byte vectors (they may span one vector more).
int kernel_class_for(int32_t max_cols, int elem_bytes, bool shifted);

// Launches the persistent kernel: n_wg workgroups of wg_threads threads.  Worker v owns items
// [d_worker_ptr[v], d_worker_ptr[v+1]); workers are workgroups, or waves when per_wave is 1.
// Each wave gets lds_floats_per_wave floats of LDS to stage long rows (0: none).  shifted
// selects the instance that reads rows not aligned to 16-byte vectors as shifted vectors (the
// plan has such slices); temporal selects ordinary (cache-resident) instead of nontemporal
// row accesses.
hipError_t launch_softmax(bsm_dtype dtype, int kernel_class, bool shifted, bool temporal,
                          const void* in, void* out, const int32_t* d_worker_ptr,
                          const bsm_item* d_items, int n_wg, int wg_threads, int per_wave,
                          int lds_floats_per_wave, void* trace, hipStream_t stream);

// The backward op under the same table: dx = y * (dy - sum(dy * y)) per row.
hipError_t launch_softmax_backward(bsm_dtype dtype, int kernel_class, bool shifted, bool temporal,
                                   const void* y, const void* dy, void* dx,
                                   const int32_t* d_worker_ptr, const bsm_item* d_items, int n_wg,
                                   int wg_threads, int per_wave, int lds_floats_per_wave,
                                   void* trace, hipStream_t stream);

// Batched matrix product under a table whose slices are the outputs C_b (m x n each, batch
// after batch): layout 0 (NT) C_b = alpha A_b B_b^T, layout 1 (NN) C_b = alpha A_b B_b; bf16
// A and B, fp32 or bf16 C.
// Matrix-product launches: threads per workgroup, LDS bytes per workgroup, the waves per SIMD
// the kernel is compiled for, and the output rows a workgroup takes per round; single_pass:
// the one-pass score softmax (layout 2, shapes for which gemm_single_pass_shape holds).
int gemm_wg_threads();
bool gemm_single_pass_shape(int n, int k);
int gemm_lds_bytes_per_wg(bool bf16_out, bool single_pass);
int gemm_waves_per_simd(bool single_pass);
int gemm_rows_per_wg(bool single_pass);

// Worker w of the table is workgroup w (gemm_wg_threads() threads, gemm_rows_per_wg() rows
// per round).  temporal: ordinary instead of nontemporal stores of C and loads of A.
// single_pass (layout 2): the one-pass form where the shape and 16-byte operands allow it,
// else the two-pass form.
hipError_t launch_gemm(int layout, bool bf16_out, bool temporal, bool single_pass, const void* a,
                       const void* b, void* c, int m, int n, int k, float alpha,
                       const int32_t* d_worker_ptr, const bsm_item* d_items, int n_wg, void* trace,
                       hipStream_t stream);

// Largest static LDS (bytes per workgroup) of a plan's instances, forward and backward.
hipError_t static_lds_bytes(bsm_dtype dtype, int kernel_class, bool shifted, int* bytes);
// Workgroups of the plan's forward instance that fit on one CU at once (registers and LDS).
hipError_t resident_wgs_per_cu(bsm_dtype dtype, int kernel_class, bool shifted, int wg_threads,
                               size_t dyn_lds_bytes, int* n);

hipError_t launch_copy(const void* src, void* dst, int64_t bytes, int n_cu, hipStream_t stream);

// Device address of `device`'s copy of the static scratch buffer of bsm_softmax_noalloc
// (BSM_NOALLOC_SCRATCH_BYTES bytes, 256-byte aligned), looked up once per device with
// hipGetSymbolAddress; `device` must be current.
hipError_t noalloc_scratch(int device, void** ptr);

}  // namespace bsm
