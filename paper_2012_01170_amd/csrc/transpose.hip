// sbc_csr_transpose: stable transpose of the neighbourhood pattern
// (Section 3.1, "Symmetry": the reverse neighbourhood is the transposed
// matrix).  Counting sort by column: per-column counts (integer atomics),
// scan, scatter of (row, edge) through per-column cursors, then every column
// is sorted by row, which makes the result independent of the order in which
// the atomics were served.
#include "common.hpp"

namespace sbc {
namespace {

// one thread per row, over the row's edges
__global__ void col_count_kernel(int32_t n_rows, int32_t n_cols, const int32_t *__restrict__ row_ptr,
                                 const int32_t *__restrict__ col_idx, int32_t *__restrict__ count) {
    int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n_rows) return;
    for (int32_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
        int32_t c = col_idx[e];
        if (c >= 0 && c < n_cols) atomicAdd(&count[c], 1);
    }
}

__global__ void col_scatter_kernel(int32_t n_rows, int32_t n_cols,
                                   const int32_t *__restrict__ row_ptr,
                                   const int32_t *__restrict__ col_idx, int32_t *__restrict__ cursor,
                                   int32_t *__restrict__ rows_tmp, int32_t *__restrict__ perm_tmp) {
    int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n_rows) return;
    for (int32_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
        int32_t c = col_idx[e];
        if (c < 0 || c >= n_cols) continue;
        int32_t pos = atomicAdd(&cursor[c], 1);
        rows_tmp[pos] = i;
        perm_tmp[pos] = e;
    }
}

struct TransposeWs {
    int32_t *count;
    int32_t *cursor;
    int32_t *rows_tmp;
    int32_t *perm_tmp;
    int64_t *total;
    void *scan_ws;
};

TransposeWs carve_transpose(void *base, int32_t n_cols, int64_t nnz, size_t *bytes) {
    Carver cv(base);
    TransposeWs w;
    w.count = cv.take<int32_t>(n_cols);
    w.cursor = cv.take<int32_t>((size_t)n_cols + 1);
    w.rows_tmp = cv.take<int32_t>(nnz);
    w.perm_tmp = cv.take<int32_t>(nnz);
    w.total = cv.take<int64_t>(1);
    w.scan_ws = cv.take<char>(scan_workspace_bytes(n_cols));
    if (bytes) *bytes = cv.used;
    return w;
}

}  // namespace
}  // namespace sbc

using namespace sbc;

extern "C" size_t sbc_transpose_workspace_size(int32_t n_cols, int64_t nnz_bound) {
    size_t bytes = 0;
    carve_transpose(nullptr, n_cols > 0 ? n_cols : 0, nnz_bound > 0 ? nnz_bound : 0, &bytes);
    return bytes;
}

extern "C" sbc_status sbc_csr_transpose(const sbc_csr *csr, int32_t *col_ptr, int32_t *row_idx,
                                        int32_t *edge_perm, void *workspace,
                                        size_t workspace_bytes, hipStream_t stream) {
    clear_error();
    if (!csr) return fail(SBC_ERR_INVALID_ARG, "csr is null");
    if (csr->n_rows < 0 || csr->n_cols < 0 || csr->nnz_bound < 0 || !csr->row_ptr ||
        (csr->nnz_bound > 0 && !csr->col_idx))
        return fail(SBC_ERR_INVALID_ARG, "malformed csr");
    if (!col_ptr || (csr->nnz_bound > 0 && (!row_idx || !edge_perm)))
        return fail(SBC_ERR_INVALID_ARG, "null output pointer");
    size_t need = 0;
    TransposeWs ws = carve_transpose(workspace, csr->n_cols, csr->nnz_bound, &need);
    if (!workspace || workspace_bytes < need)
        return fail(SBC_ERR_WORKSPACE, "workspace smaller than sbc_transpose_workspace_size()");
    const int32_t R = csr->n_rows, C = csr->n_cols;
    SBC_TRY(fill_i32(ws.count, 0, C, stream));
    if (R > 0) {
        hipLaunchKernelGGL(col_count_kernel, dim3(grid_for(R, 256)), dim3(256), 0, stream, R, C,
                           csr->row_ptr, csr->col_idx, ws.count);
        SBC_LAUNCH_CHECK();
    }
    SBC_TRY(exclusive_scan_i32(ws.count, col_ptr, C, ws.total, ws.scan_ws, stream, ws.cursor));
    if (R > 0 && C > 0) {
        hipLaunchKernelGGL(col_scatter_kernel, dim3(grid_for(R, 256)), dim3(256), 0, stream, R, C,
                           csr->row_ptr, csr->col_idx, ws.cursor, ws.rows_tmp, ws.perm_tmp);
        SBC_LAUNCH_CHECK();
        trace_before("transpose_sort", stream);
        SBC_TRY(segmented_sort_pairs(col_ptr, C, ws.rows_tmp, ws.perm_tmp, row_idx, edge_perm,
                                     stream));
        trace_after("transpose_sort", stream);
    }
    return SBC_OK;
}
