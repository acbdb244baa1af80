// Gather-accumulate over the neighbourhood pattern: the sparse products of
// the convolution (Section 3.1, N^(m) F and its transposed counterparts).
//
// One wave per output row of the pattern (a CSR row, or a CSC column for the
// transposed products); each lane owns channels c = lane, lane + 64, ...
//   expand:   out[r, m*C + c] = sum_e v[e, m] X[idx(e), c]
//   contract: out[r, c]       = sum_e sum_m v[e, m] X[idx(e), m*C + c]
// Edges are taken in pattern order and m ascending, so sums are
// deterministic.  v is the materialised [E, M] basis; through a CSC the edge's
// CSR position edge_perm[k] selects its row of v.
#include "common.hpp"
#include "spmm.hpp"

namespace sbc {
namespace {

__device__ __forceinline__ float ldx(const float *p, int64_t i) { return p[i]; }
__device__ __forceinline__ float ldx(const uint16_t *p, int64_t i) {
    return __uint_as_float((uint32_t)p[i] << 16);
}

template <int M, bool kContract, typename XT>
__global__ void __launch_bounds__(256)
    spmm_kernel(int32_t n_rows, const int32_t *__restrict__ ptr, const int32_t *__restrict__ idx,
                const int32_t *__restrict__ perm, const float *__restrict__ v,
                const XT *__restrict__ X, int32_t C, int32_t nnz, float *__restrict__ out) {
    const int lane = threadIdx.x & 63;
    const int32_t r = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (r >= n_rows) return;
    // edges past the pattern's bound (a row pointer beyond it) are not read
    int32_t e0 = ptr[r], e1 = ptr[r + 1];
    e0 = e0 < 0 ? 0 : (e0 < nnz ? e0 : nnz);
    e1 = e1 < e0 ? e0 : (e1 < nnz ? e1 : nnz);
    for (int32_t c0 = 0; c0 < C; c0 += 64) {
        const int32_t c = c0 + lane;
        const bool on = c < C;
        if (!kContract) {
            float acc[M];
#pragma unroll
            for (int m = 0; m < M; ++m) acc[m] = 0.f;
            for (int32_t e = e0; e < e1; ++e) {
                const int32_t j = idx[e];
                const int64_t ev = perm ? perm[e] : e;
                const float f = on ? ldx(X, (int64_t)j * C + c) : 0.f;
#pragma unroll
                for (int m = 0; m < M; ++m) acc[m] += v[ev * M + m] * f;
            }
            if (on) {
#pragma unroll
                for (int m = 0; m < M; ++m) out[(int64_t)r * M * C + (int64_t)m * C + c] = acc[m];
            }
        } else {
            float acc = 0.f;
            for (int32_t e = e0; e < e1; ++e) {
                const int32_t j = idx[e];
                const int64_t ev = perm ? perm[e] : e;
#pragma unroll
                for (int m = 0; m < M; ++m) {
                    const float x = on ? ldx(X, ((int64_t)j * M + m) * C + c) : 0.f;
                    acc += v[ev * M + m] * x;
                }
            }
            if (on) out[(int64_t)r * C + c] = acc;
        }
    }
}

template <int M>
sbc_status launch_m(int32_t n_rows, const int32_t *ptr, const int32_t *idx, const int32_t *perm,
                    const float *v, const void *X, bool x_bf16, int32_t C, bool contract,
                    int32_t nnz, float *out, hipStream_t stream) {
    dim3 grid(grid_for(n_rows, 4)), block(256);
#define SBC_SPMM(CONTRACT, XT)                                                                  \
    hipLaunchKernelGGL((spmm_kernel<M, CONTRACT, XT>), grid, block, 0, stream, n_rows, ptr, idx, \
                       perm, v, static_cast<const XT *>(X), C, nnz, out)
    if (contract) {
        if (x_bf16) SBC_SPMM(true, uint16_t); else SBC_SPMM(true, float);
    } else {
        if (x_bf16) SBC_SPMM(false, uint16_t); else SBC_SPMM(false, float);
    }
#undef SBC_SPMM
    SBC_LAUNCH_CHECK();
    return SBC_OK;
}

}  // namespace

sbc_status spmm(int32_t n_rows, const int32_t *ptr, const int32_t *idx, const int32_t *perm,
                const float *v, int32_t M, const void *X, bool x_bf16, int32_t C, bool contract,
                int64_t nnz_bound, float *out, hipStream_t stream, const char *trace) {
    if (n_rows <= 0 || C <= 0) return SBC_OK;
    const int32_t nnz = nnz_bound < 0 ? 0 : (nnz_bound > INT32_MAX ? INT32_MAX : (int32_t)nnz_bound);
    if (M != 4 && M != 8 && M != 10 && M != 16 && M != 24 && M != 32)
        return fail(SBC_ERR_UNSUPPORTED, "M must be 4, 8, 10, 16, 24 or 32");
    trace_before(trace, stream);
    sbc_status st;
    switch (M) {
        case 4: st = launch_m<4>(n_rows, ptr, idx, perm, v, X, x_bf16, C, contract, nnz, out, stream); break;
        case 8: st = launch_m<8>(n_rows, ptr, idx, perm, v, X, x_bf16, C, contract, nnz, out, stream); break;
        case 10: st = launch_m<10>(n_rows, ptr, idx, perm, v, X, x_bf16, C, contract, nnz, out, stream); break;
        case 16: st = launch_m<16>(n_rows, ptr, idx, perm, v, X, x_bf16, C, contract, nnz, out, stream); break;
        case 24: st = launch_m<24>(n_rows, ptr, idx, perm, v, X, x_bf16, C, contract, nnz, out, stream); break;
        default: st = launch_m<32>(n_rows, ptr, idx, perm, v, X, x_bf16, C, contract, nnz, out, stream); break;
    }
    trace_after(trace, stream);
    return st;
}

}  // namespace sbc
