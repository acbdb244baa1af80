// The event convolution's deployment form (Section 3.2, Eq. 13-15), for a
// stream fed in batches.  Every pixel x keeps z_x, the decayed sum of the
// features of its events, and tau_x, the time of its last update; an event
// reads its output from the 3 x 3 block around it before updating its own
// pixel.  With learned decays (M_v rates lambda_uv per offset u) a pixel keeps
// one sum per basis function (u, v), each decayed at its own rate; with the
// one rate 1/tau they would all be equal, and one is kept.  A batch does not wait for its own events one by one: event i's
// output is
//   sum over offsets u of W_m(u)^T [ exp(-(t_i - tau_q)/tau) z_q
//                                   + sum over batch events j < i at q of exp(-(t_i - t_j)/tau) f_j ]
// with q = x_i - u and z, tau_q the state before the batch, which is the
// recursion's value (the decays compose).  So a batch is
//   1. the batch's per-pixel lists (stream order),
//   2. G[i, m, :], the bracket above, a thread per (event, offset, 4 channels),
//   3. Y = G W on the matrix cores (the split contraction of the routes),
//   4. the state update, a thread per (pixel, 4 channels) walking the pixel's
//      batch events in order: z <- f_j + exp(-(t_j - tau_x)/tau) z, tau_x <- t_j.
// Decay factors and sums are float64; the state and G are float32.
#include "basis.hpp"
#include "common.hpp"
#include "gemm.hpp"
#include "pixel_lists.hpp"

namespace sbc {
namespace {

constexpr int kStreamThreads = 256;
constexpr int kStreamM = 8;  // the 3 x 3 offsets without the centre

// Rates of the basis functions: rates[m] (learned decays, function m = u Mv + v)
// or 1/tau for all (rates null); the state of function m is z[(q Mz + m) C]
// with Mz = M (one sum per function) or z[q C] with Mz = 1 (one for all).
struct StreamRates {
    const float *rates;
    double inv_tau;
    int32_t M, Mv, Mz;
    __device__ double rate(int32_t m) const { return rates ? (double)rates[m] : inv_tau; }
};

__global__ void __launch_bounds__(kStreamThreads)
    stream_gather_kernel(const int32_t *__restrict__ px, const int32_t *__restrict__ py,
                         const int32_t *__restrict__ t, const float *__restrict__ F, int32_t n,
                         int32_t W, int32_t H, StreamRates R, const float *__restrict__ z,
                         const int32_t *__restrict__ z_time,
                         const int32_t *__restrict__ pix_start,
                         const int32_t *__restrict__ list, const int32_t *__restrict__ list_t,
                         int32_t C, float *__restrict__ G) {
    const int32_t chunks = (C + 3) / 4;
    const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= (int64_t)n * R.M * chunks) return;
    const int32_t c0 = (int32_t)(g % chunks) * 4;
    const int32_t m = (int32_t)((g / chunks) % R.M);
    const int32_t i = (int32_t)(g / ((int64_t)chunks * R.M));
    // offset u = m / Mv of function m: row-major over the 3 x 3 block, centre skipped
    const int32_t u = m / R.Mv;
    const int k = u < 4 ? u : u + 1;
    const int32_t qx = px[i] - (k % 3 - 1), qy = py[i] - (k / 3 - 1);
    const double lam = R.rate(m);
    const int32_t zm = R.Mz == 1 ? 0 : m;
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    if (qx >= 0 && qx < W && qy >= 0 && qy < H) {
        const int32_t q = qy * W + qx;
        const double ti = (double)t[i];
        const double a = exp(-lam * (ti - (double)z_time[q]));
        const float *zq = z + ((int64_t)q * R.Mz + zm) * C;
#pragma unroll
        for (int c = 0; c < 4; ++c)
            if (c0 + c < C) acc[c] = a * (double)zq[c0 + c];
        const int32_t e1 = pix_start[q + 1];
        for (int32_t e = pix_start[q]; e < e1; ++e) {
            const int32_t j = list[e];
            if (j >= i) break;  // the list is in stream order
            const double b = exp(-lam * (ti - (double)list_t[e]));
#pragma unroll
            for (int c = 0; c < 4; ++c)
                if (c0 + c < C) acc[c] += b * (double)F[(int64_t)j * C + c0 + c];
        }
    }
    float *row = G + ((int64_t)i * R.M + m) * C;
#pragma unroll
    for (int c = 0; c < 4; ++c)
        if (c0 + c < C) row[c0 + c] = (float)acc[c];
}

// A thread per (pixel, state, 4 channels).  The threads of one pixel may sit
// in different waves, so none of them writes the pixel's time, which the
// others read: stream_time_kernel does that afterwards.
__global__ void __launch_bounds__(kStreamThreads)
    stream_update_kernel(const float *__restrict__ F, int64_t npix, StreamRates R,
                         const int32_t *__restrict__ pix_start,
                         const int32_t *__restrict__ list, const int32_t *__restrict__ list_t,
                         int32_t C, float *__restrict__ z, const int32_t *__restrict__ z_time) {
    const int32_t chunks = (C + 3) / 4;
    const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= npix * R.Mz * chunks) return;
    const int32_t c0 = (int32_t)(g % chunks) * 4;
    const int32_t zm = (int32_t)((g / chunks) % R.Mz);
    const int64_t q = g / ((int64_t)chunks * R.Mz);
    const int32_t e0 = pix_start[q], e1 = pix_start[q + 1];
    if (e0 == e1) return;
    const double lam = R.rate(zm);
    float *zq = z + (q * R.Mz + zm) * C;
    double s[4];
    double last = (double)z_time[q];
#pragma unroll
    for (int c = 0; c < 4; ++c) s[c] = c0 + c < C ? (double)zq[c0 + c] : 0.0;
    for (int32_t e = e0; e < e1; ++e) {
        const int32_t j = list[e];
        const double tj = (double)list_t[e];
        const double a = exp(-lam * (tj - last));
#pragma unroll
        for (int c = 0; c < 4; ++c)
            if (c0 + c < C) s[c] = (double)F[(int64_t)j * C + c0 + c] + a * s[c];
        last = tj;
    }
#pragma unroll
    for (int c = 0; c < 4; ++c)
        if (c0 + c < C) zq[c0 + c] = (float)s[c];
}

// tau_x <- the time of the pixel's last batch event (pixels with none keep theirs).
__global__ void __launch_bounds__(kStreamThreads)
    stream_time_kernel(int64_t npix, const int32_t *__restrict__ pix_start,
                       const int32_t *__restrict__ list_t, int32_t *__restrict__ z_time) {
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= npix) return;
    const int32_t e0 = pix_start[q], e1 = pix_start[q + 1];
    if (e0 < e1) z_time[q] = list_t[e1 - 1];
}

struct StreamWs {
    PixelLists pl;
    uint32_t *status;
    float *G;
    float *part;
};

StreamWs carve_stream(void *base, int32_t n, int64_t npix, int32_t M, int32_t C_in,
                      int32_t C_out, size_t *bytes) {
    Carver cv(base);
    StreamWs w;
    w.pl = carve_pixel_lists(cv, n, npix);
    w.status = cv.take<uint32_t>(4);
    w.G = cv.take<float>((size_t)n * M * C_in);
    w.part = cv.take<float>(gemm_workspace_floats(n, C_out, (int64_t)M * C_in));
    if (bytes) *bytes = cv.used;
    return w;
}

sbc_status check_stream(int32_t n, int32_t width, int32_t height, int32_t M, int32_t C_in,
                        int32_t C_out) {
    if (n < 0 || width <= 0 || height <= 0)
        return fail(SBC_ERR_INVALID_ARG, "n must be >= 0, width and height > 0");
    if ((int64_t)width * height >= (int64_t)INT32_MAX)
        return fail(SBC_ERR_INVALID_ARG, "width * height must be < 2^31 - 1");
    if (C_in <= 0 || C_out <= 0) return fail(SBC_ERR_INVALID_ARG, "C_in and C_out must be > 0");
    if ((int64_t)n * M * C_in >= (int64_t)INT32_MAX)
        return fail(SBC_ERR_OVERFLOW, "n * M * C_in must be < 2^31 - 1");
    if ((int64_t)width * height * (M == kStreamM ? 1 : M) * C_in >= (int64_t)INT32_MAX * 2)
        return fail(SBC_ERR_OVERFLOW, "the state has too many entries");
    return SBC_OK;
}

size_t stream_workspace(int32_t n, int32_t width, int32_t height, int32_t M, int32_t C_in,
                        int32_t C_out) {
    if (check_stream(n, width, height, M, C_in, C_out) != SBC_OK) {
        clear_error();
        return 0;
    }
    size_t bytes = 0;
    carve_stream(nullptr, n, (int64_t)width * height, M, C_in, C_out, &bytes);
    return bytes;
}

// One batch: lists, G, Y = G W, state update, times.
sbc_status stream_step(const int32_t *px, const int32_t *py, const int32_t *t, const float *F,
                       int32_t n, int32_t width, int32_t height, StreamRates R, const float *W,
                       int32_t C_in, int32_t C_out, float *z, int32_t *z_time, float *Y,
                       void *workspace, size_t workspace_bytes, hipStream_t stream) {
    if (!z || !z_time) return fail(SBC_ERR_INVALID_ARG, "the state z, z_time is null");
    if (n == 0) return SBC_OK;
    if (!px || !py || !t || !F || !W || !Y)
        return fail(SBC_ERR_INVALID_ARG, "null event, feature, weight or output array");
    const int64_t npix = (int64_t)width * height;
    size_t need = 0;
    StreamWs ws = carve_stream(workspace, n, npix, R.M, C_in, C_out, &need);
    if (!workspace || workspace_bytes < need)
        return fail(SBC_ERR_WORKSPACE, "workspace smaller than the stream's workspace size");
    const int32_t chunks = (C_in + 3) / 4;
    trace_before("stream_lists", stream);
    SBC_TRY(fill_i32(reinterpret_cast<int32_t *>(ws.status), 0, 1, stream));
    SBC_TRY(build_pixel_lists(px, py, t, n, width, height, ws.pl, ws.status, nullptr, 0, stream));
    trace_after("stream_lists", stream);
    trace_before("stream_gather", stream);
    hipLaunchKernelGGL(stream_gather_kernel,
                       dim3(grid_for((int64_t)n * R.M * chunks, kStreamThreads)),
                       dim3(kStreamThreads), 0, stream, px, py, t, F, n, width, height, R, z,
                       z_time, ws.pl.pix_start, ws.pl.list, ws.pl.list_t, C_in, ws.G);
    SBC_LAUNCH_CHECK();
    trace_after("stream_gather", stream);
    // Y [n, C_out] = G [n, M C_in] x W [M C_in, C_out]
    SBC_TRY(gemm(ws.G, false, (int64_t)R.M * C_in, 1, W, false, C_out, 1, Y, C_out, 1, n, C_out,
                 (int64_t)R.M * C_in, ws.part, stream, "stream_gemm"));
    trace_before("stream_update", stream);
    hipLaunchKernelGGL(stream_update_kernel,
                       dim3(grid_for(npix * R.Mz * chunks, kStreamThreads)),
                       dim3(kStreamThreads), 0, stream, F, npix, R, ws.pl.pix_start, ws.pl.list,
                       ws.pl.list_t, C_in, z, z_time);
    SBC_LAUNCH_CHECK();
    hipLaunchKernelGGL(stream_time_kernel, dim3(grid_for(npix, kStreamThreads)),
                       dim3(kStreamThreads), 0, stream, npix, ws.pl.pix_start, ws.pl.list_t,
                       z_time);
    SBC_LAUNCH_CHECK();
    trace_after("stream_update", stream);
    return SBC_OK;
}

}  // namespace
}  // namespace sbc

using namespace sbc;

extern "C" size_t sbc_event_stream_workspace_size(int32_t n, int32_t width, int32_t height,
                                                  int32_t C_in, int32_t C_out) {
    return stream_workspace(n, width, height, kStreamM, C_in, C_out);
}

extern "C" sbc_status sbc_event_stream_step(const int32_t *px, const int32_t *py,
                                            const int32_t *t, const float *F, int32_t n,
                                            int32_t width, int32_t height, float tau,
                                            const float *W, int32_t C_in, int32_t C_out,
                                            float *z, int32_t *z_time, float *Y,
                                            void *workspace, size_t workspace_bytes,
                                            hipStream_t stream) {
    clear_error();
    SBC_TRY(check_stream(n, width, height, kStreamM, C_in, C_out));
    if (!(tau > 0.f)) return fail(SBC_ERR_INVALID_ARG, "tau must be > 0");
    const StreamRates R{nullptr, 1.0 / (double)tau, kStreamM, 1, 1};
    return stream_step(px, py, t, F, n, width, height, R, W, C_in, C_out, z, z_time, Y, workspace,
                       workspace_bytes, stream);
}

extern "C" size_t sbc_event_stream_decays_workspace_size(int32_t n, int32_t width,
                                                         int32_t height, int32_t n_decays,
                                                         int32_t C_in, int32_t C_out) {
    if (n_decays < 1 || n_decays > 4) return 0;
    return stream_workspace(n, width, height, kStreamM * n_decays, C_in, C_out);
}

extern "C" sbc_status sbc_event_stream_step_decays(const int32_t *px, const int32_t *py,
                                                   const int32_t *t, const float *F, int32_t n,
                                                   int32_t width, int32_t height,
                                                   const float *decays, int32_t n_decays,
                                                   const float *W, int32_t C_in, int32_t C_out,
                                                   float *z, int32_t *z_time, float *Y,
                                                   void *workspace, size_t workspace_bytes,
                                                   hipStream_t stream) {
    clear_error();
    if (n_decays < 1 || n_decays > 4)
        return fail(SBC_ERR_INVALID_ARG, "n_decays must be in 1..4");
    if (!decays) return fail(SBC_ERR_INVALID_ARG, "decays is null");
    const int32_t M = kStreamM * n_decays;
    SBC_TRY(check_stream(n, width, height, M, C_in, C_out));
    const StreamRates R{decays, 0.0, M, n_decays, M};
    return stream_step(px, py, t, F, n, width, height, R, W, C_in, C_out, z, z_time, Y, workspace,
                       workspace_bytes, stream);
}
