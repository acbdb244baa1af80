// Backwards-in-time pixel-block neighbourhoods of an event stream
// (Section 3.2: a small spatial neighbourhood extending backwards in time).
//
// Pipeline (all on the caller's stream):
//   1. per-pixel event lists in stream order: the events are sorted by pixel
//      with a stable radix sort (equal pixels keep their event order), and
//      the list bounds are where each pixel's run starts; the lists carry the
//      event timestamps alongside the indices;
//   2. runs: for each pixel q of an event i's block, the events of q with
//      index < i and t >= t_i - window form one contiguous run of q's list
//      (indices and times both ascend along it), found by two bisections; the
//      count pass sums the run lengths per event;
//   3. scan -> row_ptr;
//   4. fill pass: the (2h+1)^2 runs are copied into the row one after
//      another, block pixel by block pixel (row-major around the event), so
//      a row lists its neighbours pixel by pixel, in stream order within a
//      pixel (the order of a row's entries is free: the matrix is defined
//      entry by entry).
// Steps 2 and 4 work tile by tile over the sensor, with the lists of a tile
// and its halo staged in LDS.  The transposed pattern (Section 3.1,
// "Symmetry") comes out of the same passes by the reverse search: the block
// is symmetric, so column j lists the events i > j of j's block with
// t_i <= t_j + window, again one run per pixel, in the same block order
// around j.
// Events with a pixel outside the sensor get no neighbours and are in no
// list; a decreasing timestamp raises a flag.  Neither can make a kernel
// read or write out of bounds.
#include <climits>
#include <cmath>

#include "common.hpp"

namespace sbc {
namespace {


__device__ __forceinline__ bool valid_pixel(int32_t x, int32_t y, int32_t W, int32_t H) {
    return x >= 0 && x < W && y >= 0 && y < H;
}

// Sort key of each event: its pixel, or npix (behind every pixel) for an
// event off the sensor; raises the out-of-range and unsorted flags.
__global__ void pixel_key_kernel(const int32_t *__restrict__ px, const int32_t *__restrict__ py,
                                 const int32_t *__restrict__ t, int32_t n, int32_t W, int32_t H,
                                 int32_t *__restrict__ keys, uint32_t *status) {
    const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const int32_t x = px[i], y = py[i];
    if (i > 0 && t[i] < t[i - 1]) atomicOr(status, (uint32_t)kFlagUnsorted);
    if (!valid_pixel(x, y, W, H)) {
        atomicOr(status, (uint32_t)kFlagOutOfRange);
        keys[i] = W * H;
        return;
    }
    keys[i] = y * W + x;  // < W * H < 2^31 - 1
}

// Timestamps alongside the sorted lists.  Only the first pix_start[npix]
// list slots are filled (events off the sensor are not listed).
__global__ void list_times_kernel(const int32_t *__restrict__ list, const int32_t *__restrict__ t,
                                  const int32_t *__restrict__ pix_start, int64_t npix,
                                  int32_t *__restrict__ list_t) {
    int32_t p = blockIdx.x * blockDim.x + threadIdx.x;
    if (p >= pix_start[npix]) return;
    list_t[p] = t[list[p]];
}

// In [lo, hi) of `a` (ascending), first position with a[pos] >= v.
__device__ __forceinline__ int32_t lower_bound(const int32_t *__restrict__ a, int32_t lo,
                                               int32_t hi, int32_t v) {
    while (lo < hi) {
        int32_t mid = lo + ((hi - lo) >> 1);
        if (a[mid] < v) lo = mid + 1; else hi = mid;
    }
    return lo;
}

// Tiles of tx x ty sensor pixels (at most kMaxTile x kMaxTile, sized so that
// a tile holds about as many events as a workgroup has threads).  A
// workgroup takes one tile: it stages the lists of the tile's pixels and of
// the halo around it (the block reaches half_extent pixels beyond the tile)
// in LDS, then every event of the tile's pixels finds its runs there by
// bisection, in the pattern and in its transpose, and sums them (count pass)
// or merges them into its row and its column (fill pass).  Tiles whose lists
// exceed the stage read them from global memory instead.
constexpr int kMaxTile = 8;
constexpr int kTileThreads = 256;
constexpr int kTileCap = 2048;  // list entries staged per tile

// Exclusive scan of one value per thread over the workgroup; *total gets the sum.
__device__ __forceinline__ int32_t block_excl_scan(int32_t v, int32_t *s_w, int32_t *total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int32_t incl = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int32_t y = __shfl_up(incl, d, 64);
        if (lane >= d) incl += y;
    }
    if (lane == 63) s_w[wave] = incl;
    __syncthreads();
    int32_t base = 0, sum = 0;
    for (int w = 0; w < kTileThreads / 64; ++w) {
        if (w < wave) base += s_w[w];
        sum += s_w[w];
    }
    *total = sum;
    return base + incl - v;
}

// The (kSide x kSide) runs of event i (index i, time ti) of halo pixel p: in
// the list range [s, e) of each pixel of its block, forward (kRev false) the
// entries j < i with t_j >= t_i - window, reverse the entries j > i with
// t_j <= t_i + window.  Li / Lt: list indices and times (LDS or global);
// start/len: per halo pixel, where its list begins in Li / Lt and its length.
template <int kSide, bool kRev>
__device__ __forceinline__ int32_t tile_runs(int32_t i, int32_t ti, int32_t window, int p, int HX,
                                             const int32_t *Li, const int32_t *Lt,
                                             const int32_t *start, const int32_t *len,
                                             int32_t *lo, int32_t *hi) {
    constexpr int h = kSide / 2;
    // forward: t_j >= t_i - window; reverse: t_j < t_i + window + 1; both
    // without int32 overflow
    const int64_t tmin64 = (int64_t)ti - window;
    const int32_t tmin = tmin64 < (int64_t)INT_MIN ? INT_MIN : (int32_t)tmin64;
    const int64_t tnext64 = (int64_t)ti + window + 1;
    int32_t count = 0;
#pragma unroll
    for (int k = 0; k < kSide * kSide; ++k) {
        const int q = p + (k / kSide - h) * HX + (k % kSide - h);
        const int32_t s = start[q], e = s + len[q];
        int32_t a, b;
        if constexpr (kRev) {
            a = lower_bound(Li, s, e, i + 1);  // entries with index > i
            b = tnext64 > (int64_t)INT_MAX ? e : lower_bound(Lt, a, e, (int32_t)tnext64);
        } else {
            b = lower_bound(Li, s, e, i);      // entries with index < i
            a = lower_bound(Lt, s, b, tmin);   // ... and t >= t_i - window
        }
        lo[k] = a;
        hi[k] = b;
        count += b - a;
    }
    return count;
}

// The runs, block pixel by block pixel (each run in stream order), into
// out[dst, dst + cnt), dropping writes at or past cap.
template <int K>
__device__ __forceinline__ void copy_runs(const int32_t *Li, const int32_t *lo, const int32_t *hi,
                                          int32_t *__restrict__ out, int64_t dst, int64_t cap) {
#pragma unroll
    for (int k = 0; k < K; ++k) {
        for (int32_t a = lo[k]; a < hi[k]; ++a) {
            if (dst < cap) out[dst] = Li[a];
            ++dst;
        }
    }
}

struct TileArgs {
    int32_t n, W, H, window, tx, ty, tiles_x, n_tiles;
    int32_t dirs;                          // workgroups per tile: 1, or 2 (rows, then columns)
    const int32_t *pix_start, *list, *list_t;
    int32_t *row_len, *col_len;            // count pass (col_len: null without the transpose)
    const int32_t *row_ptr, *col_ptr;      // fill pass (col_ptr: null without the transpose)
    int32_t *col_idx, *row_idx;
    int64_t cap;
};

// Every event of the tile's pixels: its row (and column) length, or its row
// (and column) entries.  c_off: prefix of the list lengths of the tile's own
// pixels (nc + 1 entries); HX: halo row length.
// dir: 0 rows and columns, 1 rows only, 2 columns only.
template <int kSide, bool kFill>
__device__ __forceinline__ void tile_events(const TileArgs &A, const int32_t *Li,
                                            const int32_t *Lt, const int32_t *start,
                                            const int32_t *len, const int32_t *c_off, int nc,
                                            int HX, int dir) {
    constexpr int h = kSide / 2;
    constexpr int K = kSide * kSide;
    const int32_t total = c_off[nc];
    for (int32_t u = threadIdx.x; u < total; u += kTileThreads) {
        int lo = 0, hi = nc - 1;  // the tile pixel holding event u: last c with c_off[c] <= u
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (c_off[mid] <= u) lo = mid; else hi = mid - 1;
        }
        const int c = lo;
        const int p = (c / A.tx + h) * HX + (c % A.tx + h);
        const int32_t a = start[p] + (u - c_off[c]);
        const int32_t i = Li[a], ti = Lt[a];
        const bool rev = kFill ? A.col_ptr != nullptr : A.col_len != nullptr;
        // the fill's output positions, loaded before the searches so that their
        // latency passes during them
        int32_t row_dst = 0, col_dst = 0;
        if constexpr (kFill) {
            if (dir != 2) row_dst = A.row_ptr[i];
            if (rev && dir != 1) col_dst = A.col_ptr[i];
        }
        int32_t rlo[K], rhi[K];
        if (dir != 2) {
            const int32_t cnt = tile_runs<kSide, false>(i, ti, A.window, p, HX, Li, Lt, start,
                                                        len, rlo, rhi);
            if constexpr (!kFill) {
                A.row_len[i] = cnt;
            } else {
                copy_runs<K>(Li, rlo, rhi, A.col_idx, row_dst, A.cap);
            }
        }
        if (rev && dir != 1) {
            const int32_t cnt_t = tile_runs<kSide, true>(i, ti, A.window, p, HX, Li, Lt, start,
                                                         len, rlo, rhi);
            if constexpr (!kFill)
                A.col_len[i] = cnt_t;
            else
                copy_runs<K>(Li, rlo, rhi, A.row_idx, col_dst, A.cap);
        }
    }
}

template <int kSide, bool kFill>
__global__ void __launch_bounds__(kTileThreads) event_tile_kernel(TileArgs A) {
    constexpr int h = kSide / 2;
    constexpr int kMaxNP = (kMaxTile + 2 * h) * (kMaxTile + 2 * h);
    static_assert(kMaxNP <= kTileThreads, "a thread per halo pixel");
    static_assert(kMaxTile * kMaxTile <= 64, "a lane per tile pixel");
    __shared__ int32_t s_start[kMaxNP], s_gstart[kMaxNP], s_len[kMaxNP];
    __shared__ int32_t s_coff[kMaxTile * kMaxTile + 1];
    __shared__ int32_t s_w[kTileThreads / 64];
    __shared__ int32_t s_idx[kTileCap], s_t[kTileCap];
    const int tid = threadIdx.x;
    const int64_t npix = (int64_t)A.W * A.H;
    // with two workgroups per tile, the first gives the tile's rows and the
    // second its columns (twice the workgroups, half of each thread's chain)
    const int32_t tile = (int32_t)blockIdx.x / A.dirs;
    const int dir = A.dirs == 1 ? 0 : 1 + (int)(blockIdx.x % A.dirs);
    if (tile == A.n_tiles) {
        // events off the sensor (sorted behind every pixel): empty rows and columns
        if constexpr (!kFill) {
            for (int32_t a = A.pix_start[npix] + tid; a < A.n; a += kTileThreads) {
                const int32_t i = A.list[a];
                A.row_len[i] = 0;
                if (A.col_len) A.col_len[i] = 0;
            }
        }
        return;
    }
    const int HX = A.tx + 2 * h, NP = HX * (A.ty + 2 * h), nc = A.tx * A.ty;
    const int32_t tx0 = (tile % A.tiles_x) * A.tx;
    const int32_t ty0 = (tile / A.tiles_x) * A.ty;
    int32_t len = 0, gs = 0;
    if (tid < NP) {
        const int32_t x = tx0 - h + tid % HX, y = ty0 - h + tid / HX;
        if (valid_pixel(x, y, A.W, A.H)) {
            const int64_t q = (int64_t)y * A.W + x;
            gs = A.pix_start[q];
            len = A.pix_start[q + 1] - gs;
        }
    }
    int32_t total;
    const int32_t off = block_excl_scan(len, s_w, &total);
    if (tid < NP) {
        s_start[tid] = off;
        s_gstart[tid] = gs;
        s_len[tid] = len;
    }
    __syncthreads();
    // the tile's own pixels: prefix of their list lengths (wave 0)
    if (tid < 64) {
        const int c = tid;
        const int32_t v = c < nc ? s_len[(c / A.tx + h) * HX + (c % A.tx + h)] : 0;
        int32_t incl = v;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int32_t y = __shfl_up(incl, d, 64);
            if (tid >= d) incl += y;
        }
        if (c < nc) s_coff[c] = incl - v;
        if (c == nc - 1) s_coff[nc] = incl;
    }
    const bool staged = total <= kTileCap;
    if (staged) {
        for (int32_t a = tid; a < total; a += kTileThreads) {
            // the halo pixel holding entry a: the last one starting at or before a
            int lo = 0, hi = NP - 1;
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (s_start[mid] <= a) lo = mid; else hi = mid - 1;
            }
            const int32_t src = s_gstart[lo] + (a - s_start[lo]);
            s_idx[a] = A.list[src];
            s_t[a] = A.list_t[src];
        }
    }
    __syncthreads();
    if (staged)
        tile_events<kSide, kFill>(A, s_idx, s_t, s_start, s_len, s_coff, nc, HX, dir);
    else
        tile_events<kSide, kFill>(A, A.list, A.list_t, s_gstart, s_len, s_coff, nc, HX, dir);
}

struct EventsWs {
    int32_t *pix_start;
    int32_t *keys;
    int32_t *sorted;
    int32_t *list;
    int32_t *list_t;
    int32_t *row_len;
    int32_t *col_len;
    int64_t *total;
    uint32_t *status;
    void *scan_ws;
    void *sort_ws;
};

EventsWs carve_events(void *base, int32_t n, int64_t npix, size_t *bytes) {
    Carver cv(base);
    EventsWs w;
    w.pix_start = cv.take<int32_t>(npix + 1);
    w.keys = cv.take<int32_t>(n);
    w.sorted = cv.take<int32_t>(n);
    w.list = cv.take<int32_t>(n);
    w.list_t = cv.take<int32_t>(n);
    w.row_len = cv.take<int32_t>(n);
    w.col_len = cv.take<int32_t>(n);
    w.total = cv.take<int64_t>(2);
    w.status = cv.take<uint32_t>(4);
    w.scan_ws = cv.take<char>(scan2_workspace_bytes(n));
    w.sort_ws = cv.take<char>(radix_sort_workspace_bytes(n));
    if (bytes) *bytes = cv.used;
    return w;
}

// Count pass (kFill false) or fill pass over all tiles, plus one workgroup
// for the events off the sensor.
template <bool kFill>
sbc_status tiles_dispatch(int32_t half_extent, const TileArgs &A, hipStream_t stream) {
    const char *name = kFill ? "events_fill" : "events_count";
    // n_tiles * dirs tile workgroups, then the one for the events off the sensor
    const dim3 grid((unsigned)((int64_t)A.n_tiles * A.dirs + 1)), block(kTileThreads);
    trace_before(name, stream);
    switch (half_extent) {
        case 0: hipLaunchKernelGGL((event_tile_kernel<1, kFill>), grid, block, 0, stream, A); break;
        case 1: hipLaunchKernelGGL((event_tile_kernel<3, kFill>), grid, block, 0, stream, A); break;
        case 2: hipLaunchKernelGGL((event_tile_kernel<5, kFill>), grid, block, 0, stream, A); break;
        case 3: hipLaunchKernelGGL((event_tile_kernel<7, kFill>), grid, block, 0, stream, A); break;
        default: return fail(SBC_ERR_UNSUPPORTED, "half_extent must be 0..3");
    }
    SBC_LAUNCH_CHECK();
    trace_after(name, stream);
    return SBC_OK;
}

// The search; with col_ptr non-null the transposed pattern too (col_ptr,
// row_idx), in the same passes over the same pixel lists.
sbc_status search_events(const int32_t *px, const int32_t *py, const int32_t *t, int32_t n,
                         int32_t width, int32_t height, int32_t half_extent, int32_t window,
                         int32_t *row_ptr, int32_t *col_idx, int32_t *col_ptr,
                         int32_t *row_idx, int64_t col_capacity, int64_t *nnz_host,
                         void *workspace, size_t workspace_bytes, hipStream_t stream) {
    if (n < 0 || width <= 0 || height <= 0)
        return fail(SBC_ERR_INVALID_ARG, "n must be >= 0, width and height > 0");
    if ((int64_t)width * height >= (int64_t)INT32_MAX)
        return fail(SBC_ERR_INVALID_ARG, "width * height must be < 2^31 - 1");
    if (half_extent < 0 || half_extent > 3)
        return fail(SBC_ERR_UNSUPPORTED, "half_extent must be 0..3");
    if (window < 0) return fail(SBC_ERR_INVALID_ARG, "window must be >= 0");
    if (!row_ptr || (n > 0 && (!px || !py || !t)))
        return fail(SBC_ERR_INVALID_ARG, "null pointer argument");
    if (col_capacity < 0 || (col_capacity > 0 && (!col_idx || (col_ptr && !row_idx))))
        return fail(SBC_ERR_INVALID_ARG, "col_idx or row_idx is null, or col_capacity < 0");
    const int64_t npix = (int64_t)width * height;
    size_t need = 0;
    EventsWs ws = carve_events(workspace, n, npix, &need);
    if (!workspace || workspace_bytes < need)
        return fail(SBC_ERR_WORKSPACE, "workspace smaller than sbc_events_workspace_size()");

    TileArgs A{};
    A.n = n;
    A.W = width;
    A.H = height;
    A.window = window;
    // square tiles holding about kTileThreads events at the stream's mean
    // density (a tile of s x s pixels, 1 <= s <= kMaxTile)
    const double per_pix = npix > 0 ? (double)n / (double)npix : 0.0;
    int side = per_pix > 0.0 ? (int)std::lround(std::sqrt(kTileThreads / per_pix)) : kMaxTile;
    side = side < 1 ? 1 : (side > kMaxTile ? kMaxTile : side);
    A.tx = A.ty = side;
    A.tiles_x = (width + side - 1) / side;
    A.n_tiles = (int32_t)((int64_t)A.tiles_x * ((height + side - 1) / side));  // <= W * H
    A.pix_start = ws.pix_start;
    A.list = ws.list;
    A.list_t = ws.list_t;
    A.cap = col_capacity;
    A.dirs = col_ptr ? 2 : 1;

    SBC_TRY(fill_i32(reinterpret_cast<int32_t *>(ws.status), 0, 1, stream));
    if (n == 0) SBC_TRY(fill_i32(ws.pix_start, 0, npix + 1, stream));
    if (n > 0) {
        hipLaunchKernelGGL(pixel_key_kernel, dim3(grid_for(n, 256)), dim3(256), 0, stream, px, py,
                           t, n, width, height, ws.keys, ws.status);
        SBC_LAUNCH_CHECK();
        // stable: each pixel's events stay in stream order
        SBC_TRY(radix_sort_pairs(ws.keys, nullptr, nullptr, n, (int32_t)npix + 1, ws.sorted,
                                 ws.list, ws.sort_ws, stream));
        SBC_TRY(segment_bounds(ws.sorted, nullptr, n, (int32_t)npix, ws.pix_start, stream));
        // listed events = pix_start[npix] <= n; the kernel is sized by n and
        // reads the true count from the end of the scan
        hipLaunchKernelGGL(list_times_kernel, dim3(grid_for(n, 256)), dim3(256), 0, stream,
                           ws.list, t, ws.pix_start, npix, ws.list_t);
        SBC_LAUNCH_CHECK();
        TileArgs C = A;
        C.row_len = ws.row_len;
        C.col_len = col_ptr ? ws.col_len : nullptr;
        SBC_TRY(tiles_dispatch<false>(half_extent, C, stream));
    }
    // row and column pointers (the column lengths are written by the same
    // count pass), in one pair of scan launches
    if (col_ptr)
        SBC_TRY(exclusive_scan2_i32(ws.row_len, row_ptr, ws.col_len, col_ptr, n, ws.total,
                                    ws.total + 1, ws.scan_ws, stream));
    else
        SBC_TRY(exclusive_scan_i32(ws.row_len, row_ptr, n, ws.total, ws.scan_ws, stream));
    if (nnz_host) {
        int64_t host[2];
        uint32_t st = 0;
        SBC_HIP_TRY(hipMemcpyAsync(host, ws.total, sizeof(host), hipMemcpyDeviceToHost, stream));
        SBC_HIP_TRY(hipMemcpyAsync(&st, ws.status, sizeof(st), hipMemcpyDeviceToHost, stream));
        SBC_HIP_TRY(hipStreamSynchronize(stream));
        *nnz_host = host[0];
        if (st & kFlagOutOfRange) return fail(SBC_ERR_OUT_OF_RANGE, "pixel outside the sensor");
        if (st & kFlagUnsorted) return fail(SBC_ERR_UNSORTED, "timestamps must be non-decreasing");
        if (host[0] > (int64_t)INT32_MAX) return fail(SBC_ERR_OVERFLOW, "2^31 or more edges");
        if (host[0] > col_capacity)
            return fail(SBC_ERR_CAPACITY, "col_capacity " + std::to_string(col_capacity) +
                                              " < E = " + std::to_string(host[0]));
    }
    if (n > 0 && col_capacity > 0) {
        TileArgs F = A;
        F.row_ptr = row_ptr;
        F.col_idx = col_idx;
        F.col_ptr = col_ptr;
        F.row_idx = col_ptr ? row_idx : nullptr;
        SBC_TRY(tiles_dispatch<true>(half_extent, F, stream));
    }
    return SBC_OK;
}

}  // namespace
}  // namespace sbc

using namespace sbc;

extern "C" size_t sbc_events_workspace_size(int32_t n, int32_t width, int32_t height) {
    size_t bytes = 0;
    int64_t npix = (int64_t)(width > 0 ? width : 0) * (height > 0 ? height : 0);
    carve_events(nullptr, n > 0 ? n : 0, npix, &bytes);
    return bytes;
}

extern "C" sbc_status sbc_neighbour_search_events(const int32_t *px, const int32_t *py,
                                                  const int32_t *t, int32_t n, int32_t width,
                                                  int32_t height, int32_t half_extent,
                                                  int32_t window, int32_t *row_ptr,
                                                  int32_t *col_idx, int64_t col_capacity,
                                                  int64_t *nnz_host, void *workspace,
                                                  size_t workspace_bytes, hipStream_t stream) {
    clear_error();
    return search_events(px, py, t, n, width, height, half_extent, window, row_ptr, col_idx,
                         nullptr, nullptr, col_capacity, nnz_host, workspace, workspace_bytes,
                         stream);
}

extern "C" sbc_status sbc_neighbour_search_events_csc(
    const int32_t *px, const int32_t *py, const int32_t *t, int32_t n, int32_t width,
    int32_t height, int32_t half_extent, int32_t window, int32_t *row_ptr, int32_t *col_idx,
    int32_t *col_ptr, int32_t *row_idx, int64_t capacity, int64_t *nnz_host, void *workspace,
    size_t workspace_bytes, hipStream_t stream) {
    clear_error();
    if (!col_ptr) return fail(SBC_ERR_INVALID_ARG, "col_ptr is null");
    return search_events(px, py, t, n, width, height, half_extent, window, row_ptr, col_idx,
                         col_ptr, row_idx, capacity, nnz_host, workspace, workspace_bytes,
                         stream);
}
