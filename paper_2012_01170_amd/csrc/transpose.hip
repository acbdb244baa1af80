// sbc_csr_transpose: stable transpose of the neighbourhood pattern
// (Section 3.1, "Symmetry": the reverse neighbourhood is the transposed
// matrix).  Counting sort by column, edge-parallel: per-column counts
// (integer atomics), scan, scatter of (row, edge, column) through per-column
// cursors, then every column is ordered by edge index (equivalently by row,
// since edge indices ascend with the row), which makes the result independent
// of the order in which the atomics were served.
//
// Edges are e in [0, min(row_ptr[n_rows], nnz_bound)), so a malformed row_ptr
// can never move a read or write outside the caller's arrays.
#include "common.hpp"

namespace sbc {
namespace {

constexpr int kScatterThreads = 256;
constexpr int kScatterItems = 4;
constexpr int kScatterChunk = kScatterThreads * kScatterItems;  // edges per block

__device__ __forceinline__ int64_t edge_count(const int32_t *row_ptr, int32_t n_rows,
                                              int64_t nnz_bound) {
    const int64_t e = row_ptr[n_rows];
    return e < 0 ? 0 : (e < nnz_bound ? e : nnz_bound);
}

// last row r in [lo, hi] with row_ptr[r] <= e (the row that holds edge e)
__device__ __forceinline__ int32_t row_of(const int32_t *__restrict__ row_ptr, int32_t lo,
                                          int32_t hi, int64_t e) {
    while (lo < hi) {
        const int32_t mid = lo + ((hi - lo + 1) >> 1);
        if ((int64_t)row_ptr[mid] <= e) lo = mid; else hi = mid - 1;
    }
    return lo;
}

__global__ void col_count_kernel(const int32_t *__restrict__ row_ptr, int32_t n_rows,
                                 int64_t nnz_bound, int32_t n_cols,
                                 const int32_t *__restrict__ col_idx, int32_t *__restrict__ count) {
    const int64_t E = edge_count(row_ptr, n_rows, nnz_bound);
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < E;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int32_t c = col_idx[e];
        if (c >= 0 && c < n_cols) atomicAdd(&count[c], 1);
    }
}

// Each block scatters kScatterChunk consecutive edges.  Two threads locate
// the rows of the chunk's first and last edges; every edge then finds its row
// by bisection between those two.
__global__ void __launch_bounds__(kScatterThreads)
    col_scatter_kernel(const int32_t *__restrict__ row_ptr, int32_t n_rows, int64_t nnz_bound,
                       int32_t n_cols, const int32_t *__restrict__ col_idx,
                       int32_t *__restrict__ cursor, int32_t *__restrict__ rows_tmp,
                       int32_t *__restrict__ perm_tmp, int32_t *__restrict__ cols_tmp) {
    __shared__ int32_t span[2];
    const int64_t E = edge_count(row_ptr, n_rows, nnz_bound);
    const int64_t e0 = (int64_t)blockIdx.x * kScatterChunk;
    if (e0 >= E) return;  // the whole block leaves together
    const int64_t e1 = e0 + kScatterChunk < E ? e0 + kScatterChunk : E;
    if (threadIdx.x < 2) span[threadIdx.x] = row_of(row_ptr, 0, n_rows - 1, threadIdx.x ? e1 - 1 : e0);
    __syncthreads();
    const int32_t r0 = span[0], r1 = span[1];
#pragma unroll
    for (int q = 0; q < kScatterItems; ++q) {
        const int64_t e = e0 + q * kScatterThreads + threadIdx.x;
        if (e >= e1) break;
        const int32_t c = col_idx[e];
        if (c < 0 || c >= n_cols) continue;
        const int32_t r = row_of(row_ptr, r0, r1, e);
        const int32_t pos = atomicAdd(&cursor[c], 1);
        rows_tmp[pos] = r;
        perm_tmp[pos] = (int32_t)e;
        cols_tmp[pos] = c;
    }
}

struct TransposeWs {
    int32_t *count;
    int32_t *cursor;
    int32_t *rows_tmp;
    int32_t *perm_tmp;
    int32_t *cols_tmp;
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
    w.cols_tmp = cv.take<int32_t>(nnz);
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
    const int64_t nnz = csr->nnz_bound;
    SBC_TRY(fill_i32(ws.count, 0, C, stream));
    if (R > 0 && nnz > 0) {
        int64_t g = (nnz + 255) / 256;
        if (g > 8192) g = 8192;
        trace_before("transpose_count", stream);
        hipLaunchKernelGGL(col_count_kernel, dim3((unsigned)g), dim3(256), 0, stream, csr->row_ptr,
                           R, nnz, C, csr->col_idx, ws.count);
        SBC_LAUNCH_CHECK();
        trace_after("transpose_count", stream);
    }
    SBC_TRY(exclusive_scan_i32(ws.count, col_ptr, C, ws.total, ws.scan_ws, stream, ws.cursor));
    if (R > 0 && C > 0 && nnz > 0) {
        const int64_t g = (nnz + kScatterChunk - 1) / kScatterChunk;
        trace_before("transpose_scatter", stream);
        hipLaunchKernelGGL(col_scatter_kernel, dim3((unsigned)g), dim3(kScatterThreads), 0, stream,
                           csr->row_ptr, R, nnz, C, csr->col_idx, ws.cursor, ws.rows_tmp,
                           ws.perm_tmp, ws.cols_tmp);
        SBC_LAUNCH_CHECK();
        trace_after("transpose_scatter", stream);
        trace_before("transpose_sort", stream);
        // key = edge index (ascends with the row), payload = row
        SBC_TRY(segmented_sort_pairs(col_ptr, C, ws.cols_tmp, nnz, ws.perm_tmp, ws.rows_tmp,
                                     edge_perm, row_idx, stream));
        trace_after("transpose_sort", stream);
    }
    return SBC_OK;
}
