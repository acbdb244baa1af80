// The leaky integrate-and-fire event sampler (the supplementary's event network
// details, and Section 4's stream hierarchy): it turns an event stream into the
// next, coarser one.  Each output cell holds a potential that decays with the
// time since its last update; every input event in its receptive field adds
// 1/n (n = how many cells that event reaches), and when the potential exceeds
// the threshold it is reset and the cell emits an event at the input's time.
//
// A cell's potential depends only on the events of its own receptive field, in
// stream order, so the cells run in parallel, a thread each:
//   1. the events are sorted by pixel (stable, so each pixel's list keeps
//      stream order), with their times alongside;
//   2. each cell merges the lists of its k x k input pixels by event index
//      (the smallest head first), advancing its potential in float64; a spike
//      of event i at the cell sets flag[i * slots + slot], slot being the
//      cell's row-major place among the cells event i reaches;
//   3. a scan over the flags gives every spike its place in the output, which
//      is thereby ordered by input event, then cell row, then cell column (the
//      sequential emission order), and a last kernel writes the events.
// The receptive field of cell (ox, oy) is the k x k block of pixels centred on
// (ox * S, oy * S) (a padded strided convolution: the output grid has
// ceil(W / S) x ceil(H / S) cells).
#include "common.hpp"

namespace sbc {
namespace {

constexpr int kLifThreads = 64;
constexpr int kLifMaxKernel = 5;

struct LifArgs {
    const int32_t *px, *py;
    int32_t n, W, H, Wo, Ho, k, S, pad, nsd;  // nsd: cells per dimension one input can reach
    double decay, thresh, reset;
    const int32_t *pix_start, *list, *list_t;
    int32_t *flags;                           // [n * nsd * nsd]
};

// Cells o (one dimension) whose receptive field [o*S - pad, o*S - pad + k)
// holds input coordinate x: lo..hi (empty when hi < lo).
__device__ __forceinline__ void cell_range(int32_t x, const LifArgs &A, int32_t n_out,
                                           int32_t &lo, int32_t &hi) {
    const int32_t a = x + A.pad - A.k + 1;  // o * S >= a
    lo = a <= 0 ? 0 : (a + A.S - 1) / A.S;
    hi = (x + A.pad) / A.S;
    hi = hi < n_out - 1 ? hi : n_out - 1;
}

__global__ void lif_key_kernel(const int32_t *__restrict__ px, const int32_t *__restrict__ py,
                               const int32_t *__restrict__ t, int32_t n, int32_t W, int32_t H,
                               int32_t *__restrict__ keys, uint32_t *status) {
    const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const int32_t x = px[i], y = py[i];
    if (i > 0 && t[i] < t[i - 1]) atomicOr(status, (uint32_t)kFlagUnsorted);
    if (x < 0 || x >= W || y < 0 || y >= H) {
        atomicOr(status, (uint32_t)kFlagOutOfRange);
        keys[i] = W * H;  // behind every pixel, seen by no cell
        return;
    }
    keys[i] = y * W + x;
}

__global__ void lif_times_kernel(const int32_t *__restrict__ list, const int32_t *__restrict__ t,
                                 int32_t n, int32_t *__restrict__ list_t) {
    const int32_t p = blockIdx.x * blockDim.x + threadIdx.x;
    if (p < n) list_t[p] = t[list[p]];
}

// One thread per output cell; K is the kernel size.
template <int K>
__global__ void __launch_bounds__(kLifThreads) lif_cell_kernel(LifArgs A) {
#pragma clang fp contract(off)
    constexpr int Q = K * K;
    constexpr int32_t kNone = INT32_MAX;
    const int32_t c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= A.Wo * A.Ho) return;
    const int32_t ox = c % A.Wo, oy = c / A.Wo;
    const int32_t x0 = ox * A.S - A.pad, y0 = oy * A.S - A.pad;
    int32_t pos[Q], end[Q], head[Q], head_t[Q], slot[Q];
    double inc[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int32_t x = x0 + q % K, y = y0 + q / K;
        pos[q] = end[q] = 0;
        slot[q] = 0;
        inc[q] = 0.0;
        if (x >= 0 && x < A.W && y >= 0 && y < A.H) {
            const int32_t p = y * A.W + x;
            pos[q] = A.pix_start[p];
            end[q] = A.pix_start[p + 1];
            int32_t lx, hx, ly, hy;
            cell_range(x, A, A.Wo, lx, hx);
            cell_range(y, A, A.Ho, ly, hy);
            // this cell is among them, so n >= 1
            inc[q] = 1.0 / (double)((hx - lx + 1) * (hy - ly + 1));
            slot[q] = (oy - ly) * A.nsd + (ox - lx);
        }
        head[q] = pos[q] < end[q] ? A.list[pos[q]] : kNone;
        head_t[q] = pos[q] < end[q] ? A.list_t[pos[q]] : 0;
    }
    const int64_t nslots = (int64_t)A.nsd * A.nsd;
    double V = 0.0, T = 0.0;
    for (;;) {
        // the earliest pending event of the receptive field
        int32_t best = kNone, bt = 0, bs = 0, bq = -1;
        double binc = 0.0;
#pragma unroll
        for (int q = 0; q < Q; ++q)
            if (head[q] < best) {
                best = head[q];
                bt = head_t[q];
                bs = slot[q];
                binc = inc[q];
                bq = q;
            }
        if (best == kNone) break;
        // advance that list (one load of the next head and its time)
        int32_t np = 0, ne = 0;
#pragma unroll
        for (int q = 0; q < Q; ++q)
            if (q == bq) {
                np = pos[q] + 1;
                ne = end[q];
            }
        const bool more = np < ne;
        const int32_t nh = more ? A.list[np] : kNone;
        const int32_t nt = more ? A.list_t[np] : 0;
#pragma unroll
        for (int q = 0; q < Q; ++q)
            if (q == bq) {
                pos[q] = np;
                head[q] = nh;
                head_t[q] = nt;
            }
        const double ti = (double)bt;
        double v = V * exp(-(ti - T) / A.decay) + binc;
        if (v > A.thresh) {
            v = A.reset;
            A.flags[(int64_t)best * nslots + bs] = 1;
        }
        V = v;
        T = ti;
    }
}

// One thread per (event, slot): the spikes, in scan order.
__global__ void lif_emit_kernel(LifArgs A, const int32_t *__restrict__ flags,
                                const int32_t *__restrict__ place, const int32_t *__restrict__ t,
                                int64_t capacity, int32_t *__restrict__ out_x,
                                int32_t *__restrict__ out_y, int32_t *__restrict__ out_t,
                                int32_t *__restrict__ out_src) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t nslots = (int64_t)A.nsd * A.nsd;
    if (e >= (int64_t)A.n * nslots || !flags[e]) return;
    const int64_t o = place[e];
    if (o >= capacity) return;
    const int32_t i = (int32_t)(e / nslots), s = (int32_t)(e % nslots);
    int32_t lx, hx, ly, hy;
    cell_range(A.px[i], A, A.Wo, lx, hx);
    cell_range(A.py[i], A, A.Ho, ly, hy);
    out_x[o] = lx + s % A.nsd;
    out_y[o] = ly + s / A.nsd;
    out_t[o] = t[i];
    if (out_src) out_src[o] = i;
}

struct LifWs {
    int32_t *keys, *sorted, *list, *list_t, *pix_start, *flags, *place;
    int64_t *total;
    uint32_t *status;
    void *scan_ws, *sort_ws;
};

int32_t lif_slots(int32_t kernel, int32_t stride) {
    const int32_t nsd = (kernel - 1) / stride + 1;
    return nsd * nsd;
}

LifWs carve_lif(void *base, int32_t n, int64_t npix, int64_t nflags, size_t *bytes) {
    Carver cv(base);
    LifWs w;
    w.keys = cv.take<int32_t>(n);
    w.sorted = cv.take<int32_t>(n);
    w.list = cv.take<int32_t>(n);
    w.list_t = cv.take<int32_t>(n);
    w.pix_start = cv.take<int32_t>(npix + 1);
    w.flags = cv.take<int32_t>(nflags);
    w.place = cv.take<int32_t>(nflags + 1);
    w.total = cv.take<int64_t>(2);
    w.status = cv.take<uint32_t>(4);
    w.scan_ws = cv.take<char>(scan_workspace_bytes(nflags));
    w.sort_ws = cv.take<char>(radix_sort_workspace_bytes(n));
    if (bytes) *bytes = cv.used;
    return w;
}

sbc_status check_lif_shape(int32_t n, int32_t width, int32_t height, int32_t kernel,
                           int32_t stride) {
    if (n < 0 || width <= 0 || height <= 0)
        return fail(SBC_ERR_INVALID_ARG, "n must be >= 0, width and height > 0");
    if ((int64_t)width * height >= (int64_t)INT32_MAX)
        return fail(SBC_ERR_INVALID_ARG, "width * height must be < 2^31 - 1");
    if (kernel < 1 || kernel > kLifMaxKernel)
        return fail(SBC_ERR_UNSUPPORTED, "kernel must be 1..5");
    if (stride < 1) return fail(SBC_ERR_INVALID_ARG, "stride must be >= 1");
    if ((int64_t)n * lif_slots(kernel, stride) >= (int64_t)INT32_MAX)
        return fail(SBC_ERR_OVERFLOW, "n * cells reached per event must be < 2^31 - 1");
    return SBC_OK;
}

}  // namespace
}  // namespace sbc

using namespace sbc;

extern "C" size_t sbc_lif_workspace_size(int32_t n, int32_t width, int32_t height,
                                         int32_t kernel, int32_t stride) {
    if (check_lif_shape(n, width, height, kernel, stride) != SBC_OK) {
        clear_error();
        return 0;
    }
    size_t bytes = 0;
    carve_lif(nullptr, n, (int64_t)width * height, (int64_t)n * lif_slots(kernel, stride),
              &bytes);
    return bytes;
}

extern "C" sbc_status sbc_lif_sample_events(const int32_t *px, const int32_t *py,
                                            const int32_t *t, int32_t n, int32_t width,
                                            int32_t height, int32_t kernel, int32_t stride,
                                            double decay, double v_thresh, double v_reset,
                                            int32_t *out_x, int32_t *out_y, int32_t *out_t,
                                            int32_t *out_src, int64_t capacity,
                                            int64_t *n_out_dev, int64_t *n_out_host,
                                            void *workspace, size_t workspace_bytes,
                                            hipStream_t stream) {
    clear_error();
    SBC_TRY(check_lif_shape(n, width, height, kernel, stride));
    if (!(decay > 0.0)) return fail(SBC_ERR_INVALID_ARG, "decay must be > 0 (inf: no decay)");
    if (n > 0 && (!px || !py || !t)) return fail(SBC_ERR_INVALID_ARG, "null event arrays");
    if (capacity < 0 || (capacity > 0 && (!out_x || !out_y || !out_t)))
        return fail(SBC_ERR_INVALID_ARG, "output arrays are null, or capacity < 0");
    const int64_t npix = (int64_t)width * height;
    const int32_t slots = lif_slots(kernel, stride);
    const int64_t nflags = (int64_t)n * slots;
    size_t need = 0;
    LifWs ws = carve_lif(workspace, n, npix, nflags, &need);
    if (!workspace || workspace_bytes < need)
        return fail(SBC_ERR_WORKSPACE, "workspace smaller than sbc_lif_workspace_size()");
    LifArgs A{};
    A.px = px;
    A.py = py;
    A.n = n;
    A.W = width;
    A.H = height;
    A.S = stride;
    A.k = kernel;
    A.pad = (kernel - 1) / 2;
    A.Wo = (width + stride - 1) / stride;
    A.Ho = (height + stride - 1) / stride;
    A.nsd = (kernel - 1) / stride + 1;
    A.decay = decay;
    A.thresh = v_thresh;
    A.reset = v_reset;
    A.pix_start = ws.pix_start;
    A.list = ws.list;
    A.list_t = ws.list_t;
    A.flags = ws.flags;
    int64_t *total = n_out_dev ? n_out_dev : ws.total;

    SBC_TRY(fill_i32(reinterpret_cast<int32_t *>(ws.status), 0, 1, stream));
    if (n > 0) {
        trace_before("lif_sort", stream);
        hipLaunchKernelGGL(lif_key_kernel, dim3(grid_for(n, 256)), dim3(256), 0, stream, px, py, t,
                           n, width, height, ws.keys, ws.status);
        SBC_LAUNCH_CHECK();
        SBC_TRY(radix_sort_pairs(ws.keys, nullptr, nullptr, n, (int32_t)npix + 1, ws.sorted,
                                 ws.list, ws.sort_ws, stream));
        SBC_TRY(segment_bounds(ws.sorted, nullptr, n, (int32_t)npix, ws.pix_start, stream));
        hipLaunchKernelGGL(lif_times_kernel, dim3(grid_for(n, 256)), dim3(256), 0, stream,
                           ws.list, t, n, ws.list_t);
        SBC_LAUNCH_CHECK();
        SBC_TRY(fill_i32(ws.flags, 0, nflags, stream));
        trace_after("lif_sort", stream);
        const int64_t cells = (int64_t)A.Wo * A.Ho;
        const dim3 grid(grid_for(cells, kLifThreads)), block(kLifThreads);
        trace_before("lif_cells", stream);
        switch (kernel) {
            case 1: hipLaunchKernelGGL(lif_cell_kernel<1>, grid, block, 0, stream, A); break;
            case 2: hipLaunchKernelGGL(lif_cell_kernel<2>, grid, block, 0, stream, A); break;
            case 3: hipLaunchKernelGGL(lif_cell_kernel<3>, grid, block, 0, stream, A); break;
            case 4: hipLaunchKernelGGL(lif_cell_kernel<4>, grid, block, 0, stream, A); break;
            default: hipLaunchKernelGGL(lif_cell_kernel<5>, grid, block, 0, stream, A); break;
        }
        SBC_LAUNCH_CHECK();
        trace_after("lif_cells", stream);
    }
    SBC_TRY(exclusive_scan_i32(ws.flags, ws.place, nflags, total, ws.scan_ws, stream));
    if (nflags > 0 && capacity > 0) {
        trace_before("lif_emit", stream);
        hipLaunchKernelGGL(lif_emit_kernel, dim3(grid_for(nflags, 256)), dim3(256), 0, stream, A,
                           ws.flags, ws.place, t, capacity, out_x, out_y, out_t, out_src);
        SBC_LAUNCH_CHECK();
        trace_after("lif_emit", stream);
    }
    if (n_out_host) {
        int64_t count = 0;
        uint32_t st = 0;
        SBC_HIP_TRY(hipMemcpyAsync(&count, total, sizeof(count), hipMemcpyDeviceToHost, stream));
        SBC_HIP_TRY(hipMemcpyAsync(&st, ws.status, sizeof(st), hipMemcpyDeviceToHost, stream));
        SBC_HIP_TRY(hipStreamSynchronize(stream));
        *n_out_host = count;
        if (st & kFlagOutOfRange) return fail(SBC_ERR_OUT_OF_RANGE, "pixel outside the sensor");
        if (st & kFlagUnsorted) return fail(SBC_ERR_UNSORTED, "timestamps must be non-decreasing");
        if (count > capacity)
            return fail(SBC_ERR_CAPACITY, "capacity " + std::to_string(capacity) +
                                              " < output events " + std::to_string(count));
    }
    return SBC_OK;
}
