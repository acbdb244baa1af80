// Dense contraction C[R, N] = A[R, K] x B[K, N] on the matrix cores (gemm.hip).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "../../include/sbconv.h"

namespace sbc {

// Number of K splits the contraction uses for this shape (1: no split).
int32_t gemm_splits(int32_t R, int32_t N, int64_t K);
// Floats of partial-tile workspace the contraction needs for this shape.
size_t gemm_workspace_floats(int32_t R, int32_t N, int64_t K);
// A(r, k) = A[r*sa_r + k*sa_k], B(k, n) = B[k*sb_k + n*sb_n],
// C(r, n) = C[r*sc_r + n*sc_n]; bf16 operands are uint16 bit patterns.
sbc_status gemm(const void *A, bool a_bf16, int64_t sa_r, int64_t sa_k, const void *B,
                bool b_bf16, int64_t sb_k, int64_t sb_n, float *C, int64_t sc_r, int64_t sc_n,
                int32_t R, int32_t N, int64_t K, float *partial_ws, hipStream_t stream,
                const char *trace);

}  // namespace sbc
