// The featureless convolution (Section 3.1, "Featureless Convolutions",
// Eq. 9-10): when every input carries the constant feature 1, the feature
// matrix drops out and Z = G~ Phi_0, where G~[i, m] adds up the values of
// basis function m along row i and Phi_0 is an M x P matrix.
//
// Forward: a group of kFLanes lanes per row takes the row's edges in turn,
// evaluates their basis values (or reads them), and adds them up in float64,
// lane partial sums first and then a butterfly, so the sums do not depend on
// scheduling; the group then writes Z[i, :] = G~[i, :] Phi_0, a lane per
// output channel.  Backward: dPhi_0 = G~^T dZ; the same kernel writes G~ into
// the workspace and the dense contraction (split over rows, summed in split
// order) multiplies it by dZ.
#include "basis.hpp"
#include "common.hpp"
#include "gemm.hpp"
#include "spmm.hpp"

namespace sbc {
namespace {

constexpr int kFLanes = 16;
constexpr int kFThreads = 256;

// kMode: 0 basis values read from v; 1 windowed point monomials; 2 event
// offsets with decay; 3 the weighted monomials (Eq. 11).
template <int M, int kMode, bool kWriteZ>
__global__ void __launch_bounds__(kFThreads)
    featureless_kernel(int32_t n_rows, const int32_t *__restrict__ row_ptr,
                       const int32_t *__restrict__ col_idx, int64_t nnz_bound,
                       const float *__restrict__ v, sbc_geometry g,
                       const float *__restrict__ Phi, int32_t P, float *__restrict__ out) {
    const int sl = threadIdx.x % kFLanes;
    const int64_t r = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kFLanes;
    if (r >= n_rows) return;  // a group leaves as a whole
    // entries past nnz_bound (a malformed pattern) are not read
    const int64_t e1 = row_ptr[r + 1] < nnz_bound ? (int64_t)row_ptr[r + 1] : nnz_bound;
    const int64_t e0 = row_ptr[r] < e1 ? (int64_t)row_ptr[r] : e1;
    const double inv_r = kMode == 1 || kMode == 3 ? 1.0 / (double)g.radius : 0.0;
    const float inv_tau = kMode == 2 ? 1.0f / g.tau : 0.f;
    float qx = 0.f, qy = 0.f, qz = 0.f;
    if constexpr (kMode == 1 || kMode == 3) {
        qx = g.x_out[3 * r];
        qy = g.x_out[3 * r + 1];
        qz = g.x_out[3 * r + 2];
    }
    // the weighted basis normalises by the row's weight sum
    double wsum = 0.0;
    if constexpr (kMode == 3) {
        for (int64_t e = e0 + sl; e < e1; e += kFLanes) {
            const int64_t j = col_idx[e];
            wsum += point_weight(qx, qy, qz, g.x_in[3 * j], g.x_in[3 * j + 1], g.x_in[3 * j + 2],
                                 inv_r);
        }
#pragma unroll
        for (int d = kFLanes / 2; d >= 1; d >>= 1) wsum += __shfl_xor(wsum, d, kFLanes);
    }
    double acc[M];
#pragma unroll
    for (int m = 0; m < M; ++m) acc[m] = 0.0;
    for (int64_t e = e0 + sl; e < e1; e += kFLanes) {
        float b[M];
        if constexpr (kMode == 0) {
#pragma unroll
            for (int m = 0; m < M; ++m) b[m] = v[e * M + m];
        } else if constexpr (kMode == 1) {
            const int64_t j = col_idx[e];
            point_basis<M>(qx, qy, qz, g.x_in[3 * j], g.x_in[3 * j + 1], g.x_in[3 * j + 2], inv_r,
                           b);
        } else if constexpr (kMode == 2) {
            const int64_t j = col_idx[e];
            const int k = event_index(g.px[r] - g.px[j], g.py[r] - g.py[j]);
            const float d = event_decay(g.t[r], g.t[j], inv_tau);
#pragma unroll
            for (int m = 0; m < M; ++m) b[m] = m == k ? d : 0.f;
        } else {
            const int64_t j = col_idx[e];
            const float px = g.x_in[3 * j], py = g.x_in[3 * j + 1], pz = g.x_in[3 * j + 2];
            const double w = point_weight(qx, qy, qz, px, py, pz, inv_r);
            weighted_mono10(qx, qy, qz, px, py, pz, inv_r, wsum != 0.0 ? w / wsum : 0.0, b);
        }
#pragma unroll
        for (int m = 0; m < M; ++m) acc[m] += (double)b[m];
    }
#pragma unroll
    for (int d = kFLanes / 2; d >= 1; d >>= 1)
#pragma unroll
        for (int m = 0; m < M; ++m) acc[m] += __shfl_xor(acc[m], d, kFLanes);
    if constexpr (!kWriteZ) {
        if (sl < M) {
            float gm = 0.f;
#pragma unroll
            for (int m = 0; m < M; ++m)
                if (m == sl) gm = (float)acc[m];
            out[r * M + sl] = gm;
        }
    } else {
        for (int32_t p = sl; p < P; p += kFLanes) {
            double z = 0.0;
#pragma unroll
            for (int m = 0; m < M; ++m) z += acc[m] * (double)Phi[(int64_t)m * P + p];
            out[r * P + p] = (float)z;
        }
    }
}

template <bool kWriteZ>
sbc_status launch_featureless(const sbc_csr *csr, const float *v, const sbc_geometry *g,
                              int32_t M, const float *Phi, int32_t P, float *out,
                              hipStream_t stream) {
    const dim3 grid(grid_for((int64_t)csr->n_rows * kFLanes, kFThreads)), block(kFThreads);
    const int mode = v ? 0
                       : g->basis == SBC_BASIS_EVENT8 ? 2
                       : g->basis == SBC_BASIS_WMONO10 ? 3 : 1;
    const sbc_geometry gg = g ? *g : sbc_geometry{};
#define SBC_FL(MM, MODE)                                                                        \
    hipLaunchKernelGGL((featureless_kernel<MM, MODE, kWriteZ>), grid, block, 0, stream,          \
                       csr->n_rows, csr->row_ptr, csr->col_idx, csr->nnz_bound, v, gg, Phi, P, \
                       out)
    if (mode == 0) {
        if (M == 4) SBC_FL(4, 0); else if (M == 8) SBC_FL(8, 0); else SBC_FL(10, 0);
    } else if (mode == 1) {
        if (M == 4) SBC_FL(4, 1); else SBC_FL(8, 1);
    } else if (mode == 2) {
        SBC_FL(8, 2);
    } else {
        SBC_FL(10, 3);
    }
#undef SBC_FL
    SBC_LAUNCH_CHECK();
    return SBC_OK;
}

sbc_status check_featureless(const sbc_csr *csr, const float *v, const sbc_geometry *g,
                             int32_t M, int32_t P) {
    SBC_TRY(check_csr(csr));
    if (M != 4 && M != 8 && M != 10) return fail(SBC_ERR_UNSUPPORTED, "M must be 4, 8 or 10");
    if (P <= 0) return fail(SBC_ERR_INVALID_ARG, "P must be > 0");
    if (!v) {
        SBC_TRY(check_geometry(g, csr->n_rows, csr->n_cols));
        if (g->basis == SBC_BASIS_EVENT_DECAYS)
            return fail(SBC_ERR_UNSUPPORTED, "the learned-decay basis needs v here");
        if (sbc_basis_size(g->basis) != M)
            return fail(SBC_ERR_INVALID_ARG, "M does not match the geometry's basis");
    }
    return SBC_OK;
}

}  // namespace
}  // namespace sbc

using namespace sbc;

extern "C" size_t sbc_featureless_workspace_size(int32_t n_out, int32_t M, int32_t P) {
    if (n_out < 0 || M <= 0 || P <= 0) return 0;
    return align_up((size_t)n_out * M * 4) + gemm_workspace_floats(M, P, n_out) * 4;
}

extern "C" sbc_status sbc_featureless_forward(const sbc_csr *csr, const float *v,
                                              const sbc_geometry *geometry, int32_t M,
                                              const float *Phi, int32_t P, float *Z,
                                              hipStream_t stream) {
    clear_error();
    SBC_TRY(check_featureless(csr, v, geometry, M, P));
    if (csr->n_rows == 0) return SBC_OK;
    if (!Phi || !Z) return fail(SBC_ERR_INVALID_ARG, "Phi or Z is null");
    trace_before("featureless_fwd", stream);
    SBC_TRY(launch_featureless<true>(csr, v, geometry, M, Phi, P, Z, stream));
    trace_after("featureless_fwd", stream);
    return SBC_OK;
}

extern "C" sbc_status sbc_featureless_backward(const sbc_csr *csr, const float *v,
                                               const sbc_geometry *geometry, int32_t M,
                                               const float *dZ, int32_t P, float *dPhi,
                                               void *workspace, size_t workspace_bytes,
                                               hipStream_t stream) {
    clear_error();
    SBC_TRY(check_featureless(csr, v, geometry, M, P));
    if (!dPhi) return fail(SBC_ERR_INVALID_ARG, "dPhi is null");
    const int32_t n = csr->n_rows;
    if (n > 0 && !dZ) return fail(SBC_ERR_INVALID_ARG, "dZ is null");
    const size_t need = sbc_featureless_workspace_size(n, M, P);
    if (!workspace || workspace_bytes < need)
        return fail(SBC_ERR_WORKSPACE, "workspace smaller than sbc_featureless_workspace_size()");
    if (n == 0) return fill_i32(reinterpret_cast<int32_t *>(dPhi), 0, (int64_t)M * P, stream);
    float *Gt = static_cast<float *>(workspace);
    float *part = reinterpret_cast<float *>(static_cast<char *>(workspace) +
                                            align_up((size_t)n * M * 4));
    trace_before("featureless_rowsum", stream);
    SBC_TRY(launch_featureless<false>(csr, v, geometry, M, nullptr, P, Gt, stream));
    trace_after("featureless_rowsum", stream);
    // dPhi [M, P] = G~^T [M, n] x dZ [n, P]
    return gemm(Gt, false, 1, M, dZ, false, P, 1, dPhi, P, 1, M, P, n, part, stream,
                "featureless_dphi");
}
