// sbc_basis_eval: materialise the values v[E, M] of the neighbourhood matrices
// (Section 3.1, the entries of N^(m)).  One wave per group of 64 rows would
// scatter the writes; instead every thread takes one edge and finds its row by
// binary search in row_ptr, so that the [E, M] rows are written contiguously.
#include "basis.hpp"
#include "common.hpp"

namespace sbc {

__device__ __forceinline__ int32_t row_of_edge(const int32_t *__restrict__ row_ptr,
                                               int32_t n_rows, int32_t e) {
    int32_t lo = 0, hi = n_rows;  // row_ptr[lo] <= e < row_ptr[hi]
    while (hi - lo > 1) {
        int32_t mid = (lo + hi) >> 1;
        if (row_ptr[mid] <= e) lo = mid; else hi = mid;
    }
    return lo;
}

// Values of the entries of a compressed pattern in its own entry order: a CSR
// (segments = outputs i, indices = inputs j) or, with kT, its transpose
// (segments = inputs j, indices = outputs i).
template <int kBasis, bool kT>
__global__ void __launch_bounds__(256)
    basis_kernel(int32_t n_seg, const int32_t *__restrict__ seg_ptr,
                 const int32_t *__restrict__ idx, int64_t nnz_bound, sbc_geometry g,
                 float *__restrict__ v) {
    constexpr int M = kBasis == SBC_BASIS_MONO4 ? 4 : 8;
    // entries past nnz_bound (a malformed pattern) have no room in v
    const int64_t E = seg_ptr[n_seg] < nnz_bound ? (int64_t)seg_ptr[n_seg] : nnz_bound;
    const double inv_r = 1.0 / (double)g.radius;
    const float inv_tau = 1.0f / g.tau;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < E;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int32_t sg = row_of_edge(seg_ptr, n_seg, (int32_t)e);
        const int32_t other = idx[e];
        const int32_t i = kT ? other : sg;
        const int32_t j = kT ? sg : other;
        float out[8];
        if constexpr (kBasis == SBC_BASIS_EVENT8) {
#pragma unroll
            for (int m = 0; m < 8; ++m) out[m] = 0.f;
            const int k = event_index(g.px[i] - g.px[j], g.py[i] - g.py[j]);
            const float d = event_decay(g.t[i], g.t[j], inv_tau);
#pragma unroll
            for (int m = 0; m < 8; ++m)
                if (m == k) out[m] = d;
        } else {
            point_basis<M>(g.x_out[3 * (int64_t)i], g.x_out[3 * (int64_t)i + 1],
                           g.x_out[3 * (int64_t)i + 2], g.x_in[3 * (int64_t)j],
                           g.x_in[3 * (int64_t)j + 1], g.x_in[3 * (int64_t)j + 2], inv_r, out);
        }
#pragma unroll
        for (int m = 0; m < M; ++m) v[e * M + m] = out[m];
    }
}

// Learned-decay event values (Eq. 12 with n_decays rates per offset), in the
// entry order of a CSR or (kT) of its transpose: zero except the n_decays
// entries of the edge's offset, exp(-lambda dt), or with kDeriv their
// derivatives with respect to lambda, -dt exp(-lambda dt).
template <bool kT, bool kDeriv>
__global__ void __launch_bounds__(256)
    decay_basis_kernel(int32_t n_seg, const int32_t *__restrict__ seg_ptr,
                       const int32_t *__restrict__ idx, int64_t nnz_bound, sbc_geometry g,
                       float *__restrict__ v) {
    const int Mv = g.n_decays, M = 8 * Mv;
    const int64_t E = seg_ptr[n_seg] < nnz_bound ? (int64_t)seg_ptr[n_seg] : nnz_bound;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < E;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int32_t sg = row_of_edge(seg_ptr, n_seg, (int32_t)e);
        const int32_t other = idx[e];
        const int32_t i = kT ? other : sg;
        const int32_t j = kT ? sg : other;
        const int k = event_index(g.px[i] - g.px[j], g.py[i] - g.py[j]);
        const float dt = (float)((int64_t)g.t[i] - (int64_t)g.t[j]);
        for (int m = 0; m < M; ++m) v[e * M + m] = 0.f;
        if (k >= 0) {
            for (int q = 0; q < Mv; ++q) {
                const float x = expf(-g.decays[k * Mv + q] * dt);
                v[e * M + k * Mv + q] = kDeriv ? -dt * x : x;
            }
        }
    }
}

// Weighted values (Eq. 11): a group of kWLanes lanes per row sums the row's
// weights in float64 (lane partial sums in edge order, then a butterfly, so
// the sum does not depend on scheduling) and writes every edge's ten values
// times w / W_i; the row's [E, 10] values are contiguous.
constexpr int kWLanes = 16;

__global__ void __launch_bounds__(256)
    weighted_basis_kernel(int32_t n_rows, const int32_t *__restrict__ row_ptr,
                          const int32_t *__restrict__ col_idx, int64_t nnz_bound, sbc_geometry g,
                          float *__restrict__ v) {
    const int sl = threadIdx.x % kWLanes;
    const int64_t r = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWLanes;
    if (r >= n_rows) return;  // a group leaves as a whole
    // entries past nnz_bound (a malformed pattern) have no room in v
    int64_t e1 = row_ptr[r + 1] < nnz_bound ? (int64_t)row_ptr[r + 1] : nnz_bound;
    int64_t e0 = row_ptr[r] < e1 ? (int64_t)row_ptr[r] : e1;
    const double inv_r = 1.0 / (double)g.radius;
    const float qx = g.x_out[3 * r], qy = g.x_out[3 * r + 1], qz = g.x_out[3 * r + 2];
    double wsum = 0.0;
    for (int64_t e = e0 + sl; e < e1; e += kWLanes) {
        const int64_t j = col_idx[e];
        wsum += point_weight(qx, qy, qz, g.x_in[3 * j], g.x_in[3 * j + 1], g.x_in[3 * j + 2], inv_r);
    }
#pragma unroll
    for (int d = kWLanes / 2; d >= 1; d >>= 1) wsum += __shfl_xor(wsum, d, kWLanes);
    for (int64_t e = e0 + sl; e < e1; e += kWLanes) {
        const int64_t j = col_idx[e];
        const float px = g.x_in[3 * j], py = g.x_in[3 * j + 1], pz = g.x_in[3 * j + 2];
        const double w = point_weight(qx, qy, qz, px, py, pz, inv_r);
        const double s = wsum != 0.0 ? w / wsum : 0.0;
        float out[10];
        weighted_mono10(qx, qy, qz, px, py, pz, inv_r, s, out);
#pragma unroll
        for (int m = 0; m < 10; ++m) v[e * 10 + m] = out[m];
    }
}

sbc_status check_geometry(const sbc_geometry *g, int32_t n_rows, int32_t n_cols) {
    if (!g) return fail(SBC_ERR_INVALID_ARG, "geometry is null");
    switch (g->basis) {
        case SBC_BASIS_MONO4:
        case SBC_BASIS_MONO8:
        case SBC_BASIS_WMONO10:
            if (!(g->radius > 0.f)) return fail(SBC_ERR_INVALID_ARG, "radius must be > 0");
            if ((n_rows > 0 && !g->x_out) || (n_cols > 0 && !g->x_in))
                return fail(SBC_ERR_INVALID_ARG, "x_in / x_out is null");
            return SBC_OK;
        case SBC_BASIS_EVENT_DECAYS:
            if (g->n_decays < 2 || g->n_decays > 4 || !g->decays)
                return fail(SBC_ERR_INVALID_ARG, "n_decays must be 2..4 with decays non-null");
            if (n_rows != n_cols)
                return fail(SBC_ERR_INVALID_ARG, "event streams are in place (n_rows == n_cols)");
            if (n_rows > 0 && (!g->px || !g->py || !g->t))
                return fail(SBC_ERR_INVALID_ARG, "px / py / t is null");
            return SBC_OK;
        case SBC_BASIS_EVENT8:
            if (!(g->tau > 0.f)) return fail(SBC_ERR_INVALID_ARG, "tau must be > 0");
            if (n_rows != n_cols)
                return fail(SBC_ERR_INVALID_ARG, "event streams are in place (n_rows == n_cols)");
            if (n_rows > 0 && (!g->px || !g->py || !g->t))
                return fail(SBC_ERR_INVALID_ARG, "px / py / t is null");
            return SBC_OK;
        default:
            return fail(SBC_ERR_INVALID_ARG, "unknown basis");
    }
}

template <bool kT>
sbc_status basis_launch(int32_t n_seg, const int32_t *seg_ptr, const int32_t *idx, int64_t nnz,
                        const sbc_geometry *g, float *v, hipStream_t stream) {
    if (n_seg == 0 || nnz <= 0) return SBC_OK;
    if (g->basis == SBC_BASIS_WMONO10) {
        // normalised by row sums: only in CSR order
        if (kT) return fail(SBC_ERR_UNSUPPORTED, "the weighted basis is evaluated in CSR order");
        trace_before("basis", stream);
        hipLaunchKernelGGL(weighted_basis_kernel, dim3(grid_for((int64_t)n_seg * kWLanes, 256)),
                           dim3(256), 0, stream, n_seg, seg_ptr, idx, nnz, *g, v);
        SBC_LAUNCH_CHECK();
        trace_after("basis", stream);
        return SBC_OK;
    }
    int64_t blocks = (nnz + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    if (g->basis == SBC_BASIS_EVENT_DECAYS) {
        trace_before("basis", stream);
        hipLaunchKernelGGL((decay_basis_kernel<kT, false>), dim3((unsigned)blocks), dim3(256), 0,
                           stream, n_seg, seg_ptr, idx, nnz, *g, v);
        SBC_LAUNCH_CHECK();
        trace_after("basis", stream);
        return SBC_OK;
    }
    trace_before("basis", stream);
    switch (g->basis) {
        case SBC_BASIS_MONO4:
            hipLaunchKernelGGL((basis_kernel<SBC_BASIS_MONO4, kT>), dim3((unsigned)blocks),
                               dim3(256), 0, stream, n_seg, seg_ptr, idx, nnz, *g, v);
            break;
        case SBC_BASIS_MONO8:
            hipLaunchKernelGGL((basis_kernel<SBC_BASIS_MONO8, kT>), dim3((unsigned)blocks),
                               dim3(256), 0, stream, n_seg, seg_ptr, idx, nnz, *g, v);
            break;
        default:
            hipLaunchKernelGGL((basis_kernel<SBC_BASIS_EVENT8, kT>), dim3((unsigned)blocks),
                               dim3(256), 0, stream, n_seg, seg_ptr, idx, nnz, *g, v);
            break;
    }
    SBC_LAUNCH_CHECK();
    trace_after("basis", stream);
    return SBC_OK;
}

sbc_status basis_eval_launch(const sbc_csr *csr, const sbc_geometry *g, float *v,
                             hipStream_t stream) {
    return basis_launch<false>(csr->n_rows, csr->row_ptr, csr->col_idx, csr->nnz_bound, g, v,
                               stream);
}

sbc_status decay_derivative_launch(const sbc_csr *csr, const sbc_geometry *g, float *v,
                                   hipStream_t stream) {
    if (csr->n_rows == 0 || csr->nnz_bound <= 0) return SBC_OK;
    int64_t blocks = (csr->nnz_bound + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    trace_before("decay_basis", stream);
    hipLaunchKernelGGL((decay_basis_kernel<false, true>), dim3((unsigned)blocks), dim3(256), 0,
                       stream, csr->n_rows, csr->row_ptr, csr->col_idx, csr->nnz_bound, *g, v);
    SBC_LAUNCH_CHECK();
    trace_after("decay_basis", stream);
    return SBC_OK;
}

sbc_status basis_eval_t_launch(const sbc_csc *csc, int64_t nnz_bound, const sbc_geometry *g,
                               float *v, hipStream_t stream) {
    return basis_launch<true>(csc->n_cols, csc->col_ptr, csc->row_idx, nnz_bound, g, v, stream);
}

sbc_status check_csr(const sbc_csr *csr) {
    if (!csr) return fail(SBC_ERR_INVALID_ARG, "csr is null");
    if (csr->n_rows < 0 || csr->n_cols < 0 || csr->nnz_bound < 0)
        return fail(SBC_ERR_INVALID_ARG, "negative csr size");
    if (csr->nnz_bound > (int64_t)INT32_MAX) return fail(SBC_ERR_OVERFLOW, "2^31 or more edges");
    if (!csr->row_ptr || (csr->nnz_bound > 0 && !csr->col_idx))
        return fail(SBC_ERR_INVALID_ARG, "csr row_ptr / col_idx is null");
    return SBC_OK;
}

}  // namespace sbc

using namespace sbc;

extern "C" sbc_status sbc_basis_eval(const sbc_csr *csr, const sbc_geometry *geometry, float *v,
                                     hipStream_t stream) {
    clear_error();
    SBC_TRY(check_csr(csr));
    SBC_TRY(check_geometry(geometry, csr->n_rows, csr->n_cols));
    if (csr->nnz_bound > 0 && !v) return fail(SBC_ERR_INVALID_ARG, "v is null");
    return basis_eval_launch(csr, geometry, v, stream);
}
