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
//      (indices and times both ascend along it); for blocks up to 3x3 the
//      runs of all events come from one two-pointer sweep per (pixel,
//      offset) pair and are stored, for larger blocks each event bisects;
//      the count pass sums the run lengths per event;
//   3. scan -> row_ptr;
//   4. fill pass: the (2h+1)^2 runs are merged by index into the row.
// The transposed pattern (Section 3.1, "Symmetry") comes from the same lists
// by the reverse search: the block is symmetric, so column j lists the events
// i > j of j's block with t_i <= t_j + window, again one run per pixel.
// Events with a pixel outside the sensor get no neighbours and are in no
// list; a decreasing timestamp raises a flag.  Neither can make a kernel
// read or write out of bounds.
#include <climits>

#include "common.hpp"

namespace sbc {
namespace {

constexpr int kMaxBlock = 7;  // half_extent <= 3: at most 7x7 pixels

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

struct Runs {
    int32_t lo[kMaxBlock * kMaxBlock];
    int32_t hi[kMaxBlock * kMaxBlock];
};

// Runs of event i in the lists of its block's pixels.  Forward: the events
// j < i with t_j >= t_i - window; reverse (kRev): the events j > i with
// t_j <= t_i + window.
template <int kSide, bool kRev>
__device__ __forceinline__ int32_t find_runs(int32_t i, int32_t x, int32_t y, int32_t ti,
                                             int32_t W, int32_t H, int64_t window,
                                             const int32_t *__restrict__ pix_start,
                                             const int32_t *__restrict__ list,
                                             const int32_t *__restrict__ list_t, Runs &r) {
    constexpr int h = kSide / 2;
    // forward: t_j >= t_i - window; reverse: t_j < t_i + window + 1; both
    // without int32 overflow
    const int64_t tmin64 = (int64_t)ti - window;
    const int32_t tmin = tmin64 < (int64_t)INT_MIN ? INT_MIN : (int32_t)tmin64;
    const int64_t tnext64 = (int64_t)ti + window + 1;
    int32_t count = 0;
#pragma unroll
    for (int k = 0; k < kSide * kSide; ++k) {
        const int32_t qx = x + (k % kSide) - h, qy = y + (k / kSide) - h;
        int32_t lo = 0, hi = 0;
        if (valid_pixel(qx, qy, W, H)) {
            const int64_t q = (int64_t)qy * W + qx;
            const int32_t s = pix_start[q], e = pix_start[q + 1];
            if constexpr (kRev) {
                lo = lower_bound(list, s, e, i + 1);  // entries with index > i
                hi = tnext64 > (int64_t)INT_MAX ? e : lower_bound(list_t, lo, e, (int32_t)tnext64);
            } else {
                hi = lower_bound(list, s, e, i);        // entries with index < i
                lo = lower_bound(list_t, s, hi, tmin);  // ... and t >= t_i - window
            }
        }
        r.lo[k] = lo;
        r.hi[k] = hi;
        count += hi - lo;
    }
    return count;
}

// Runs of every event in the lists of its block's pixels, by a two-pointer
// sweep: one thread per (pixel p, offset k) walks the events of p in stream
// order.  For event i the run in the list of q = p + offset is [lo, hi).
// Forward: hi is the first entry with index >= i and lo the first with
// t >= t_i - window.  Reverse (kRev): lo is the first entry with index > i
// and hi the first at or after lo with t > t_i + window.  Every bound only
// moves forward as i grows (indices and times ascend along every list), so
// each list is read once per thread instead of bisected per event.
// runs[i * kRunsK + k] = (lo, hi); offsets past the sensor give (0, 0).
constexpr int kRunsK = 9;  // stored runs per event: blocks up to 3x3

template <int kSide, bool kRev>
__global__ void pixel_runs_kernel(int64_t npix, int32_t W, int32_t H, int32_t window,
                                  const int32_t *__restrict__ pix_start,
                                  const int32_t *__restrict__ list,
                                  const int32_t *__restrict__ list_t, int2 *__restrict__ runs) {
    constexpr int K = kSide * kSide;
    constexpr int h = kSide / 2;
    static_assert(K <= kRunsK, "runs are stored for blocks up to 3x3");
    const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (tid >= npix * K) return;
    const int64_t p = tid / K;
    const int k = (int)(tid % K);
    const int32_t x = (int32_t)(p % W), y = (int32_t)(p / W);
    const int32_t qx = x + (k % kSide) - h, qy = y + (k / kSide) - h;
    const int32_t ps = pix_start[p], pe = pix_start[p + 1];
    if (!valid_pixel(qx, qy, W, H)) {
        for (int32_t a = ps; a < pe; ++a) runs[(int64_t)list[a] * kRunsK + k] = make_int2(0, 0);
        return;
    }
    const int64_t q = (int64_t)qy * W + qx;
    const int32_t qe = pix_start[q + 1];
    int32_t lo = pix_start[q], hi = lo;
    for (int32_t a = ps; a < pe; ++a) {
        const int32_t i = list[a];
        if constexpr (kRev) {
            // t_j <= t_i + window, computed without int32 overflow
            const int64_t tmax = (int64_t)list_t[a] + window;
            while (lo < qe && list[lo] <= i) ++lo;
            if (hi < lo) hi = lo;
            while (hi < qe && (int64_t)list_t[hi] <= tmax) ++hi;
        } else {
            // t_j >= t_i - window, computed without int32 overflow
            const int64_t tmin64 = (int64_t)list_t[a] - window;
            const int32_t tmin = tmin64 < (int64_t)INT_MIN ? INT_MIN : (int32_t)tmin64;
            while (hi < qe && list[hi] < i) ++hi;
            while (lo < hi && list_t[lo] < tmin) ++lo;
        }
        runs[(int64_t)i * kRunsK + k] = make_int2(lo, hi);
    }
}

// kStored: runs read from pixel_runs_kernel's output, else found by bisection.
// kRev: the reverse search (rows of the transposed pattern).
template <int kSide, bool kStored, bool kRev>
__global__ void __launch_bounds__(256)
    event_rows_kernel(const int32_t *__restrict__ px, const int32_t *__restrict__ py,
                      const int32_t *__restrict__ t, int32_t n, int32_t W, int32_t H,
                      int32_t window, const int32_t *__restrict__ pix_start,
                      const int32_t *__restrict__ list, const int32_t *__restrict__ list_t,
                      int32_t *__restrict__ row_len, const int32_t *__restrict__ row_ptr,
                      int32_t *__restrict__ col_idx, int64_t col_capacity,
                      const int2 *__restrict__ runs) {
    const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const int32_t x = px[i], y = py[i];
    if (!valid_pixel(x, y, W, H)) {
        if (row_len) row_len[i] = 0;
        return;
    }
    Runs r;
    int32_t cnt = 0;
    if constexpr (kStored) {
#pragma unroll
        for (int k = 0; k < kSide * kSide; ++k) {
            const int2 lh = runs[(int64_t)i * kRunsK + k];
            r.lo[k] = lh.x;
            r.hi[k] = lh.y;
            cnt += lh.y - lh.x;
        }
    } else {
        cnt = find_runs<kSide, kRev>(i, x, y, t[i], W, H, (int64_t)window, pix_start, list, list_t, r);
    }
    if (row_len) {
        row_len[i] = cnt;
        return;
    }
    // merge the runs by event index (each run ascends; runs are disjoint)
    int64_t dst = row_ptr[i];
    int32_t head[kSide * kSide];
#pragma unroll
    for (int k = 0; k < kSide * kSide; ++k) head[k] = r.lo[k] < r.hi[k] ? list[r.lo[k]] : INT_MAX;
    for (int32_t out = 0; out < cnt; ++out) {
        int32_t best = INT_MAX, arg = 0;
#pragma unroll
        for (int k = 0; k < kSide * kSide; ++k) {
            if (head[k] < best) {
                best = head[k];
                arg = k;
            }
        }
#pragma unroll
        for (int k = 0; k < kSide * kSide; ++k) {
            if (k == arg) {
                ++r.lo[k];
                head[k] = r.lo[k] < r.hi[k] ? list[r.lo[k]] : INT_MAX;
            }
        }
        if (dst < col_capacity) col_idx[dst] = best;
        ++dst;
    }
}

struct EventsWs {
    int32_t *pix_start;
    int32_t *keys;
    int32_t *sorted;
    int32_t *list;
    int32_t *list_t;
    int32_t *row_len;
    int2 *runs;
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
    w.runs = cv.take<int2>((size_t)n * kRunsK);
    w.total = cv.take<int64_t>(2);
    w.status = cv.take<uint32_t>(4);
    w.scan_ws = cv.take<char>(scan_workspace_bytes(n));
    w.sort_ws = cv.take<char>(radix_sort_workspace_bytes(n));
    if (bytes) *bytes = cv.used;
    return w;
}

template <int kSide, bool kRev>
void launch_rows(int32_t n, const int32_t *px, const int32_t *py, const int32_t *t, int32_t W,
                 int32_t H, int32_t window, const EventsWs &ws, int32_t *row_len,
                 const int32_t *row_ptr, int32_t *col_idx, int64_t cap, hipStream_t stream) {
    constexpr bool kStored = kSide * kSide <= kRunsK;
    hipLaunchKernelGGL((event_rows_kernel<kSide, kStored, kRev>), dim3(grid_for(n, 256)),
                       dim3(256), 0, stream, px, py, t, n, W, H, window, ws.pix_start, ws.list,
                       ws.list_t, row_len, row_ptr, col_idx, cap, ws.runs);
}

template <int kSide, bool kRev>
void launch_runs(int64_t npix, int32_t W, int32_t H, int32_t window, const EventsWs &ws,
                 hipStream_t stream) {
    if constexpr (kSide * kSide <= kRunsK) {
        const int64_t threads = npix * kSide * kSide;
        hipLaunchKernelGGL((pixel_runs_kernel<kSide, kRev>),
                           dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, stream, npix, W,
                           H, window, ws.pix_start, ws.list, ws.list_t, ws.runs);
    }
}

template <bool kRev>
sbc_status runs_dispatch(int32_t half_extent, int64_t npix, int32_t W, int32_t H, int32_t window,
                         const EventsWs &ws, hipStream_t stream) {
    switch (half_extent) {
        case 0: launch_runs<1, kRev>(npix, W, H, window, ws, stream); break;
        case 1: launch_runs<3, kRev>(npix, W, H, window, ws, stream); break;
        default: return SBC_OK;  // larger blocks bisect per event
    }
    SBC_LAUNCH_CHECK();
    return SBC_OK;
}

// Count pass (row_len != null; computes the runs first) or fill pass, of the
// pattern (kRev false) or of its transpose (kRev true).
template <bool kRev>
sbc_status rows_dispatch(int32_t half_extent, int64_t npix, int32_t n, const int32_t *px,
                         const int32_t *py, const int32_t *t, int32_t W, int32_t H,
                         int32_t window, const EventsWs &ws, int32_t *row_len,
                         const int32_t *row_ptr, int32_t *col_idx, int64_t cap,
                         hipStream_t stream) {
    const char *name = kRev ? (row_len ? "events_count_t" : "events_fill_t")
                            : (row_len ? "events_count" : "events_fill");
    trace_before(name, stream);
    if (row_len) SBC_TRY(runs_dispatch<kRev>(half_extent, npix, W, H, window, ws, stream));
    switch (half_extent) {
        case 0: launch_rows<1, kRev>(n, px, py, t, W, H, window, ws, row_len, row_ptr, col_idx, cap, stream); break;
        case 1: launch_rows<3, kRev>(n, px, py, t, W, H, window, ws, row_len, row_ptr, col_idx, cap, stream); break;
        case 2: launch_rows<5, kRev>(n, px, py, t, W, H, window, ws, row_len, row_ptr, col_idx, cap, stream); break;
        case 3: launch_rows<7, kRev>(n, px, py, t, W, H, window, ws, row_len, row_ptr, col_idx, cap, stream); break;
        default: return fail(SBC_ERR_UNSUPPORTED, "half_extent must be 0..3");
    }
    SBC_LAUNCH_CHECK();
    trace_after(name, stream);
    return SBC_OK;
}

// The search; with col_ptr non-null the transposed pattern too (col_ptr,
// row_idx, from the same pixel lists, after the pattern itself).
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
        SBC_TRY(rows_dispatch<false>(half_extent, npix, n, px, py, t, width, height, window, ws,
                                     ws.row_len, nullptr, nullptr, 0, stream));
    }
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
    if (n > 0 && col_capacity > 0)
        SBC_TRY(rows_dispatch<false>(half_extent, npix, n, px, py, t, width, height, window, ws,
                                     nullptr, row_ptr, col_idx, col_capacity, stream));
    if (!col_ptr) return SBC_OK;
    // the transpose: the runs and row lengths of the pattern are no longer needed
    if (n > 0)
        SBC_TRY(rows_dispatch<true>(half_extent, npix, n, px, py, t, width, height, window, ws,
                                    ws.row_len, nullptr, nullptr, 0, stream));
    SBC_TRY(exclusive_scan_i32(ws.row_len, col_ptr, n, ws.total, ws.scan_ws, stream));
    if (n > 0 && col_capacity > 0)
        SBC_TRY(rows_dispatch<true>(half_extent, npix, n, px, py, t, width, height, window, ws,
                                    nullptr, col_ptr, row_idx, col_capacity, stream));
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
