// sbc_csr_transpose: stable transpose of the neighbourhood pattern
// (Section 3.1, "Symmetry": the reverse neighbourhood is the transposed
// matrix): each column lists its rows in ascending order, with edge_perm
// giving every entry's CSR position.  Two ways, chosen by size, both
// independent of scheduling:
//   - up to kRadixMin edges, a counting sort: per-column counts and
//     per-column cursors with integer atomics, then every column ordered by
//     edge index with a per-entry rank sort (few launches);
//   - beyond, a stable radix sort of the edges by column (values: the edge
//     indices), with no atomics, whose passes read and write in runs (global
//     atomics are served past the L2 cache here, one at a time per address,
//     which is what limits the counting sort on millions of edges).
//
// Edges are e in [0, min(row_ptr[n_rows], nnz_bound)); column indices outside
// [0, n_cols) are left out (counting sort) or sorted behind every column
// (radix sort), so a malformed pattern can never move a read or write
// outside the caller's arrays.
#include "common.hpp"

namespace sbc {
namespace {

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

constexpr int kScatterThreads = 256;
constexpr int kScatterItems = 4;
constexpr int kScatterChunk = kScatterThreads * kScatterItems;  // edges per block
// row_ptr entries a block stages in LDS for the row lookup of its edges
constexpr int kSpanMax = 2048;

// Rows of a block's edges [e0, e1): two threads locate the rows of the first
// and last edge; when the span r0..r1 is short (the usual case) its row
// bounds are staged in LDS and every edge bisects there, else in row_ptr.
struct ChunkRows {
    int32_t r0, r1;
    bool staged;
};

__device__ __forceinline__ ChunkRows chunk_rows(const int32_t *__restrict__ row_ptr,
                                                int32_t n_rows, int64_t e0, int64_t e1,
                                                int32_t *span, int32_t *s_ptr) {
    if (threadIdx.x < 2) span[threadIdx.x] = row_of(row_ptr, 0, n_rows - 1, threadIdx.x ? e1 - 1 : e0);
    __syncthreads();
    ChunkRows c{span[0], span[1], span[1] - span[0] + 1 <= kSpanMax};
    if (c.staged)
        for (int32_t k = threadIdx.x; k <= c.r1 - c.r0; k += blockDim.x) s_ptr[k] = row_ptr[c.r0 + k];
    __syncthreads();
    return c;
}

// the row holding edge e of the chunk
__device__ __forceinline__ int32_t chunk_row(const ChunkRows &c, const int32_t *__restrict__ row_ptr,
                                             const int32_t *s_ptr, int64_t e) {
    if (!c.staged) return row_of(row_ptr, c.r0, c.r1, e);
    int32_t lo = 0, hi = c.r1 - c.r0;
    while (lo < hi) {
        const int32_t mid = lo + ((hi - lo + 1) >> 1);
        if ((int64_t)s_ptr[mid] <= e) lo = mid; else hi = mid - 1;
    }
    return c.r0 + lo;
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

// Each block scatters kScatterChunk consecutive edges, each finding its row
// by bisection between the rows of the chunk's first and last edges (in LDS
// when that span is short).
__global__ void __launch_bounds__(kScatterThreads)
    col_scatter_kernel(const int32_t *__restrict__ row_ptr, int32_t n_rows, int64_t nnz_bound,
                       int32_t n_cols, const int32_t *__restrict__ col_idx,
                       int32_t *__restrict__ cursor, int32_t *__restrict__ rows_tmp,
                       int32_t *__restrict__ perm_tmp, int32_t *__restrict__ cols_tmp) {
    __shared__ int32_t span[2];
    __shared__ int32_t s_ptr[kSpanMax];
    const int64_t E = edge_count(row_ptr, n_rows, nnz_bound);
    const int64_t e0 = (int64_t)blockIdx.x * kScatterChunk;
    if (e0 >= E) return;  // the whole block leaves together
    const int64_t e1 = e0 + kScatterChunk < E ? e0 + kScatterChunk : E;
    const ChunkRows cr = chunk_rows(row_ptr, n_rows, e0, e1, span, s_ptr);
#pragma unroll
    for (int q = 0; q < kScatterItems; ++q) {
        const int64_t e = e0 + q * kScatterThreads + threadIdx.x;
        if (e >= e1) break;
        const int32_t c = col_idx[e];
        if (c < 0 || c >= n_cols) continue;
        const int32_t r = chunk_row(cr, row_ptr, s_ptr, e);
        const int32_t pos = atomicAdd(&cursor[c], 1);
        rows_tmp[pos] = r;
        perm_tmp[pos] = (int32_t)e;
        cols_tmp[pos] = c;
    }
}

// Sort keys (column, or n_cols for an invalid one) per edge, and the edge count.
__global__ void col_keys_kernel(const int32_t *__restrict__ row_ptr, int32_t n_rows,
                                int64_t nnz_bound, int32_t n_cols,
                                const int32_t *__restrict__ col_idx, int32_t *__restrict__ keys,
                                int64_t *__restrict__ n_edges) {
    const int64_t E = edge_count(row_ptr, n_rows, nnz_bound);
    const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (tid == 0) *n_edges = E;
    for (int64_t e = tid; e < E; e += (int64_t)gridDim.x * blockDim.x) {
        const int32_t c = col_idx[e];
        keys[e] = (c >= 0 && c < n_cols) ? c : n_cols;
    }
}


// rowof[e] = the row holding edge e.  Each block takes 1024 consecutive
// edges; every edge bisects between the rows of the chunk's first and last
// edge (in LDS when that span is short).
__global__ void __launch_bounds__(256)
    edge_rows_kernel(const int32_t *__restrict__ row_ptr, int32_t n_rows, int64_t nnz_bound,
                     int32_t *__restrict__ rowof) {
    __shared__ int32_t span[2];
    __shared__ int32_t s_ptr[kSpanMax];
    const int64_t E = edge_count(row_ptr, n_rows, nnz_bound);
    const int64_t e0 = (int64_t)blockIdx.x * 1024;
    if (e0 >= E) return;  // the whole block leaves together
    const int64_t e1 = e0 + 1024 < E ? e0 + 1024 : E;
    const ChunkRows cr = chunk_rows(row_ptr, n_rows, e0, e1, span, s_ptr);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int64_t e = e0 + q * 256 + threadIdx.x;
        if (e < e1) rowof[e] = chunk_row(cr, row_ptr, s_ptr, e);
    }
}

// row_idx[p] = rowof[edge_perm[p]] for the sorted positions p
__global__ void gather_rows_kernel(const int32_t *__restrict__ edge_perm,
                                   const int64_t *__restrict__ n_edges,
                                   const int32_t *__restrict__ rowof,
                                   int32_t *__restrict__ row_idx) {
    const int64_t E = *n_edges;
    for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < E;
         p += (int64_t)gridDim.x * blockDim.x)
        row_idx[p] = rowof[edge_perm[p]];
}

// Rows of the transpose workspace; the counting sort uses count, cursor and
// the three tmp arrays, the radix sort keys, sorted, rowof and sort_ws.
constexpr int64_t kRadixMin = 1 << 21;

struct TransposeWs {
    int32_t *count, *cursor, *rows_tmp, *perm_tmp, *cols_tmp;   // counting sort
    int32_t *keys, *sorted, *rowof;                               // radix sort
    int64_t *n_edges;
    void *scan_ws, *sort_ws;
};

TransposeWs carve_transpose(void *base, int32_t n_cols, int64_t nnz, size_t *bytes) {
    Carver cv(base);
    TransposeWs w{};
    w.n_edges = cv.take<int64_t>(1);
    if (nnz < kRadixMin) {
        w.count = cv.take<int32_t>(n_cols);
        w.cursor = cv.take<int32_t>((size_t)n_cols + 1);
        w.rows_tmp = cv.take<int32_t>(nnz);
        w.perm_tmp = cv.take<int32_t>(nnz);
        w.cols_tmp = cv.take<int32_t>(nnz);
        w.scan_ws = cv.take<char>(scan_workspace_bytes(n_cols));
    } else {
        w.keys = cv.take<int32_t>(nnz);
        w.sorted = cv.take<int32_t>(nnz);
        w.rowof = cv.take<int32_t>(nnz);
        w.sort_ws = cv.take<char>(radix_sort_workspace_bytes(nnz));
    }
    if (bytes) *bytes = cv.used;
    return w;
}

// ---------------------------------------------------------------- batched
// Transpose of a block-diagonal pattern (block b: rows row_splits[b] ..
// row_splits[b+1]-1, columns col_splits[b] .. col_splits[b+1]-1): the block's
// entries occupy the same positions [e0, e1) in the CSC as in the CSR, so the
// blocks are independent.  Each block's columns are cut into `slices`
// consecutive ranges, one workgroup each; a workgroup finds where its slice
// starts by counting the block's entries in the columns before it, so the
// workgroups need no communication.  A workgroup takes its slice's columns
// in windows of at most kBWin: it counts the
// window's entries per column (LDS atomics), scans the counts, stages every
// entry (edge, row) at its column's slot, orders each column by edge index
// (rank within the column) and writes the window out.  A window whose
// entries exceed the stage is halved; a single column that still does not
// fit is compacted in edge order by one wave.
constexpr int kBThreads = 512;
constexpr int kBWin = 2048;      // columns per window
constexpr int kBStage = 4096;    // staged entries per window
constexpr int kBRows = 2048;     // row bounds staged in LDS
constexpr int kBPer = 16;        // column indices a thread keeps in registers
// blocks of up to kBThreads * kBPer entries read their column indices once

__device__ __forceinline__ int32_t bisect_le(const int32_t *a, int32_t lo, int32_t hi, int64_t x) {
    // last k in [lo, hi] with a[k] <= x (a ascending, a[lo] <= x)
    while (lo < hi) {
        const int32_t mid = lo + ((hi - lo + 1) >> 1);
        if ((int64_t)a[mid] <= x) lo = mid; else hi = mid - 1;
    }
    return lo;
}

// exclusive scan of cnt[0..n) into start[0..n) by the workgroup (n <=
// 4 * kBThreads); returns the total
static_assert(kBWin <= 4 * kBThreads, "one scan step per window");
__device__ int32_t block_scan_counts(const int32_t *cnt, int32_t *start, int32_t n,
                                     int32_t *wsum) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int base = threadIdx.x * 4;
    int32_t v[4], s = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        v[k] = base + k < n ? cnt[base + k] : 0;
        s += v[k];
    }
    int32_t x = s;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int32_t y = __shfl_up(x, d, 64);
        if (lane >= d) x += y;
    }
    if (lane == 63) wsum[wave] = x;
    __syncthreads();
    int32_t before = 0, total = 0;
#pragma unroll
    for (int w = 0; w < kBThreads / 64; ++w) {
        const int32_t t = wsum[w];
        before += w < wave ? t : 0;
        total += t;
    }
    int32_t run = before + x - s;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        if (base + k < n) start[base + k] = run;
        run += v[k];
    }
    __syncthreads();
    return total;
}

__global__ void __launch_bounds__(kBThreads)
    batched_transpose_kernel(const int32_t *__restrict__ row_ptr, int32_t n_rows,
                             int64_t nnz_bound, int32_t n_cols,
                             const int32_t *__restrict__ col_idx,
                             const int32_t *__restrict__ row_splits,
                             const int32_t *__restrict__ col_splits, int32_t n_batch,
                             int32_t slices, int32_t *__restrict__ col_ptr,
                             int32_t *__restrict__ row_idx, int32_t *__restrict__ edge_perm) {
    __shared__ int32_t cnt[kBWin];
    __shared__ int32_t start[kBWin];
    __shared__ int32_t st_edge[kBStage];
    __shared__ int32_t st_row[kBStage];
    __shared__ int32_t s_rp[kBRows + 1];
    __shared__ int32_t wsum[kBThreads / 64];
    __shared__ int32_t win_e[kBStage];  // the window's entries, in no order
    __shared__ int32_t n_win;
    const int b = blockIdx.x / slices, sl = blockIdx.x % slices;
    const int tid = threadIdx.x;
    auto clampi = [](int64_t x, int64_t lo, int64_t hi) {
        return (int32_t)(x < lo ? lo : (x > hi ? hi : x));
    };
    const int64_t E = edge_count(row_ptr, n_rows, nnz_bound);
    const int32_t r0 = clampi(row_splits[b], 0, n_rows);
    const int32_t r1 = clampi(row_splits[b + 1], r0, n_rows);
    const int32_t cb0 = clampi(col_splits[b], 0, n_cols);
    const int32_t cb1 = clampi(col_splits[b + 1], cb0, n_cols);
    // this workgroup's slice of the block's columns
    const int32_t c0 = cb0 + (int32_t)((int64_t)(cb1 - cb0) * sl / slices);
    const int32_t c1 = cb0 + (int32_t)((int64_t)(cb1 - cb0) * (sl + 1) / slices);
    const int64_t e0 = clampi(row_ptr[r0], 0, E);
    const int64_t e1 = clampi(row_ptr[r1], e0, E);
    const bool rows_staged = r1 - r0 + 1 <= kBRows;
    if (rows_staged)
        for (int32_t k = tid; k <= r1 - r0; k += kBThreads) s_rp[k] = row_ptr[r0 + k];
    __syncthreads();
    auto row_of_edge = [&](int64_t e) -> int32_t {
        return rows_staged ? r0 + bisect_le(s_rp, 0, r1 - r0, e) : row_of(row_ptr, r0, r1, e);
    };
    // the block's entries as (edge, column): from registers when they fit
    const bool cached = e1 - e0 <= (int64_t)kBThreads * kBPer;
    int32_t cc[kBPer];
    if (cached) {
#pragma unroll
        for (int k = 0; k < kBPer; ++k) {
            const int64_t e = e0 + tid + (int64_t)k * kBThreads;
            cc[k] = e < e1 ? col_idx[e] : -1;
        }
    }
    auto for_edges = [&](auto &&fn) {
        if (cached) {
#pragma unroll
            for (int k = 0; k < kBPer; ++k) {
                const int64_t e = e0 + tid + (int64_t)k * kBThreads;
                if (e < e1) fn(e, cc[k]);
            }
        } else {
            for (int64_t e = e0 + tid; e < e1; e += kBThreads) fn(e, col_idx[e]);
        }
    };

    // the block's entries in the columns before the slice
    int32_t below = 0;
    if (c0 > cb0) for_edges([&](int64_t, int32_t c) { below += (c >= cb0 && c < c0) ? 1 : 0; });
    for (int d = 1; d < 64; d <<= 1) below += __shfl_xor(below, d, 64);
    if ((tid & 63) == 0) wsum[tid >> 6] = below;
    __syncthreads();
    int64_t done = 0;  // entries of this block before the next window
#pragma unroll
    for (int w = 0; w < kBThreads / 64; ++w) done += wsum[w];
    __syncthreads();
    int32_t cw = c0;
    int32_t W = c1 - cw < kBWin ? c1 - cw : kBWin;
    while (cw < c1) {
        if (W > c1 - cw) W = c1 - cw;
        for (int32_t k = tid; k < W; k += kBThreads) cnt[k] = 0;
        if (tid == 0) n_win = 0;
        __syncthreads();
        // count the window's entries per column and list them (while the
        // list fits; a window that overflows it is halved below)
        for_edges([&](int64_t e, int32_t c) {
            if (c >= cw && c < cw + W) {
                atomicAdd(&cnt[c - cw], 1);
                const int32_t q = atomicAdd(&n_win, 1);
                if (q < kBStage) win_e[q] = (int32_t)(e - e0);
            }
        });
        __syncthreads();
        const int32_t total = block_scan_counts(cnt, start, W, wsum);
        if (total > kBStage && W > 1) {  // too many entries: halve the window
            W = (W + 1) / 2;
            continue;
        }
        for (int32_t k = tid; k < W; k += kBThreads)
            col_ptr[cw + k] = (int32_t)(e0 + done + start[k]);
        if (total > kBStage) {
            // one column with more entries than the stage: wave 0 writes them
            // in edge order
            if (tid < 64) {
                int64_t out = e0 + done;
                for (int64_t eb = e0; eb < e1; eb += 64) {
                    const int64_t e = eb + tid;
                    const bool hit = e < e1 && col_idx[e] == cw;
                    const uint64_t m = __ballot(hit);
                    if (hit) {
                        const int64_t o = out + __popcll(m & ((1ull << tid) - 1ull));
                        row_idx[o] = row_of_edge(e);
                        edge_perm[o] = (int32_t)e;
                    }
                    out += __popcll(m);
                }
            }
        } else {
            // stage every listed entry at its column's slot (any order within
            // the column): one listed entry per thread and step, so the row
            // lookups do not diverge over entries outside the window
            for (int32_t k = tid; k < W; k += kBThreads) cnt[k] = 0;
            __syncthreads();
            for (int32_t q = tid; q < total; q += kBThreads) {
                const int64_t e = e0 + win_e[q];
                const int32_t c = col_idx[e];
                const int32_t slot = start[c - cw] + atomicAdd(&cnt[c - cw], 1);
                st_edge[slot] = (int32_t)e;
                st_row[slot] = row_of_edge(e);
            }
            __syncthreads();
            // order each column by edge index: an entry's rank among its column's
            for (int32_t q = tid; q < total; q += kBThreads) {
                const int32_t k = bisect_le(start, 0, W - 1, q);  // column of slot q
                const int32_t lo = start[k], hi = lo + cnt[k];
                const int32_t me = st_edge[q];
                int32_t rank = 0;
                for (int32_t t = lo; t < hi; ++t) rank += st_edge[t] < me ? 1 : 0;
                const int64_t o = e0 + done + lo + rank;
                row_idx[o] = st_row[q];
                edge_perm[o] = me;
            }
        }
        __syncthreads();
        done += total;
        cw += W;
        W = kBWin;
    }
    // the end pointer (and any columns past the last block's range)
    if (b == n_batch - 1 && sl == slices - 1)
        for (int32_t k = c1 + tid; k <= n_cols; k += kBThreads) col_ptr[k] = (int32_t)(e0 + done);
}

int grid_cap(int64_t n, int cap) {
    int64_t g = (n + 255) / 256;
    return (int)(g < 1 ? 1 : (g > cap ? cap : g));
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
    if (R == 0 || nnz == 0) return fill_i32(col_ptr, 0, (int64_t)C + 1, stream);
    if (C == INT32_MAX) return fail(SBC_ERR_INVALID_ARG, "n_cols must be < 2^31 - 1");
    if (nnz < kRadixMin) {
        SBC_TRY(fill_i32(ws.count, 0, C, stream));
        trace_before("transpose_count", stream);
        hipLaunchKernelGGL(col_count_kernel, dim3(grid_cap(nnz, 8192)), dim3(256), 0, stream,
                           csr->row_ptr, R, nnz, C, csr->col_idx, ws.count);
        SBC_LAUNCH_CHECK();
        trace_after("transpose_count", stream);
        SBC_TRY(exclusive_scan_i32(ws.count, col_ptr, C, ws.n_edges, ws.scan_ws, stream,
                                   ws.cursor));
        trace_before("transpose_scatter", stream);
        hipLaunchKernelGGL(col_scatter_kernel, dim3((unsigned)((nnz + kScatterChunk - 1) / kScatterChunk)),
                           dim3(kScatterThreads), 0, stream, csr->row_ptr, R, nnz, C,
                           csr->col_idx, ws.cursor, ws.rows_tmp, ws.perm_tmp, ws.cols_tmp);
        SBC_LAUNCH_CHECK();
        trace_after("transpose_scatter", stream);
        trace_before("transpose_sort", stream);
        // key = edge index (ascends with the row), payload = row
        SBC_TRY(segmented_sort_pairs(col_ptr, C, ws.cols_tmp, nnz, ws.perm_tmp, ws.rows_tmp,
                                     edge_perm, row_idx, stream));
        trace_after("transpose_sort", stream);
        return SBC_OK;
    }
    trace_before("transpose_count", stream);
    hipLaunchKernelGGL(col_keys_kernel, dim3(grid_cap(nnz, 8192)), dim3(256), 0, stream,
                       csr->row_ptr, R, nnz, C, csr->col_idx, ws.keys, ws.n_edges);
    SBC_LAUNCH_CHECK();
    hipLaunchKernelGGL(edge_rows_kernel, dim3((unsigned)((nnz + 1023) / 1024)), dim3(256), 0,
                       stream, csr->row_ptr, R, nnz, ws.rowof);
    SBC_LAUNCH_CHECK();
    trace_after("transpose_count", stream);
    trace_before("transpose_scatter", stream);
    // values are the edge indices: they become edge_perm
    SBC_TRY(radix_sort_pairs(ws.keys, nullptr, ws.n_edges, nnz, C + 1, ws.sorted, edge_perm,
                             ws.sort_ws, stream));
    trace_after("transpose_scatter", stream);
    trace_before("transpose_sort", stream);
    SBC_TRY(segment_bounds(ws.sorted, ws.n_edges, nnz, C, col_ptr, stream));
    hipLaunchKernelGGL(gather_rows_kernel, dim3(grid_cap(nnz, 8192)), dim3(256), 0, stream,
                       edge_perm, ws.n_edges, ws.rowof, row_idx);
    SBC_LAUNCH_CHECK();
    trace_after("transpose_sort", stream);
    return SBC_OK;
}

extern "C" sbc_status sbc_csr_transpose_batched(const sbc_csr *csr, const int32_t *row_splits,
                                                const int32_t *col_splits, int32_t n_batch,
                                                int32_t *col_ptr, int32_t *row_idx,
                                                int32_t *edge_perm, hipStream_t stream) {
    clear_error();
    if (!csr) return fail(SBC_ERR_INVALID_ARG, "csr is null");
    if (csr->n_rows < 0 || csr->n_cols < 0 || csr->nnz_bound < 0 || !csr->row_ptr ||
        (csr->nnz_bound > 0 && !csr->col_idx))
        return fail(SBC_ERR_INVALID_ARG, "malformed csr");
    if (n_batch < 1 || !row_splits || !col_splits)
        return fail(SBC_ERR_INVALID_ARG, "n_batch must be >= 1 with row and column splits");
    if (!col_ptr || (csr->nnz_bound > 0 && (!row_idx || !edge_perm)))
        return fail(SBC_ERR_INVALID_ARG, "null output pointer");
    if (csr->n_cols == INT32_MAX) return fail(SBC_ERR_INVALID_ARG, "n_cols must be < 2^31 - 1");
    if (csr->n_rows == 0 || csr->n_cols == 0 || csr->nnz_bound == 0)
        return fill_i32(col_ptr, 0, (int64_t)csr->n_cols + 1, stream);
    // about two workgroups per CU (the LDS of two fits), at least one per
    // block, at most one column per workgroup on average
    int64_t slices = (2 * (int64_t)device_cus() + n_batch - 1) / n_batch;
    const int64_t per_col = csr->n_cols / n_batch;
    if (slices > per_col) slices = per_col;
    if (slices < 1) slices = 1;
    if ((int64_t)n_batch * slices > INT32_MAX) slices = 1;
    trace_before("transpose_batched", stream);
    hipLaunchKernelGGL(batched_transpose_kernel, dim3((unsigned)(n_batch * slices)),
                       dim3(kBThreads), 0, stream, csr->row_ptr, csr->n_rows, csr->nnz_bound,
                       csr->n_cols, csr->col_idx, row_splits, col_splits, n_batch,
                       (int32_t)slices, col_ptr, row_idx, edge_perm);
    SBC_LAUNCH_CHECK();
    trace_after("transpose_batched", stream);
    return SBC_OK;
}
