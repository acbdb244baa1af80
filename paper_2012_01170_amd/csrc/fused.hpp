// Fused forward / backward kernels (fused.hip).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "../../include/sbconv.h"

namespace sbc {

// Upper bound on the persistent blocks of the fused backward (one per CU).
constexpr int kMaxBlocksBwd = 256;

bool fused_forward_available(int32_t M, int32_t CI, int32_t CO, bool bf);
bool fused_backward_available(int32_t M, int32_t CI, int32_t CO, bool bf);
// n_points: the larger of the input and output counts
size_t fused_workspace_bytes(int32_t M, int32_t CI, int32_t CO, int32_t n_points, int64_t nnz);
// the same for the forward alone (no dW partials)
size_t fused_forward_workspace_bytes(int32_t M, int32_t CI, int32_t CO, int32_t n_points,
                                     int64_t nnz);

// Y = sum_m N^(m) F W^(m) in one kernel (plus a small weight re-layout for bf16).
sbc_status fused_forward(const sbc_csr *csr, const float *v, const sbc_geometry *g, int32_t M,
                         const void *F, const void *W, bool bf, int32_t CI, int32_t CO, float *Y,
                         void *ws, hipStream_t stream);

// dF and/or dW (either may be null) by the transposed gather D = N^T dY.
sbc_status fused_backward(const sbc_csr *csr, const sbc_csc *csc, const float *v,
                          const sbc_geometry *g, int32_t M, const void *F, const void *W,
                          const void *dY, bool bf, int32_t CI, int32_t CO, float *dF, float *dW,
                          void *ws, hipStream_t stream, bool decay_derivative = false);

}  // namespace sbc
