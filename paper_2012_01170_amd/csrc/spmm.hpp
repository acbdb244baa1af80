// Gather-accumulate kernels over the neighbourhood pattern (spmm.hip).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "../../include/sbconv.h"

namespace sbc {

// Rows r < n_rows of the pattern (ptr [n_rows + 1], idx [E]); perm maps a
// pattern position to its row of v (nullptr: identity).  Expand writes
// out [n_rows, M*C]; contract reads X [*, M*C] and writes out [n_rows, C].
// Row extents are clamped to [0, nnz_bound] (the sizes idx and v were given).
sbc_status spmm(int32_t n_rows, const int32_t *ptr, const int32_t *idx, const int32_t *perm,
                const float *v, int32_t M, const void *X, bool x_bf16, int32_t C, bool contract,
                int64_t nnz_bound, float *out, hipStream_t stream, const char *trace);

// basis.hip
sbc_status check_csr(const sbc_csr *csr);
sbc_status check_geometry(const sbc_geometry *g, int32_t n_rows, int32_t n_cols);
sbc_status basis_eval_launch(const sbc_csr *csr, const sbc_geometry *g, float *v,
                             hipStream_t stream);
// the learned-decay basis's derivatives with respect to the rates (CSR order)
sbc_status decay_derivative_launch(const sbc_csr *csr, const sbc_geometry *g, float *v,
                                   hipStream_t stream);
// the same values for the entries of the transpose, in its entry order
sbc_status basis_eval_t_launch(const sbc_csc *csc, int64_t nnz_bound, const sbc_geometry *g,
                               float *v, hipStream_t stream);

}  // namespace sbc
