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
//
// The gathers are latency-bound (a few edges per row, a few rows per wave
// slot), so a wave fetches its row's columns and basis rows 64 edges at a
// time, one edge per lane, and then keeps a group of edges' feature loads in
// flight at once (edge_group) instead of one edge's.
#include "common.hpp"
#include "spmm.hpp"

namespace sbc {
namespace {

__device__ __forceinline__ float ldx(const float *p, int64_t i) { return p[i]; }
__device__ __forceinline__ float ldx(const uint16_t *p, int64_t i) {
    return __uint_as_float((uint32_t)p[i] << 16);
}

// Edges per group of loads in flight: each lane holds one float per edge and
// channel block for the expansion and M of them for the contraction.
template <int M, bool kContract>
constexpr int edge_group() {
    if (kContract) return M >= 32 ? 1 : 32 / M;
    return M >= 64 ? 1 : (64 / M > 8 ? 8 : 64 / M);
}

template <int M, bool kContract, typename XT>
__global__ void __launch_bounds__(256)
    spmm_kernel(int32_t n_rows, const int32_t *__restrict__ ptr, const int32_t *__restrict__ idx,
                const int32_t *__restrict__ perm, const float *__restrict__ v,
                const XT *__restrict__ X, int32_t C, int32_t nnz, float *__restrict__ out) {
    constexpr int U = edge_group<M, kContract>();
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
        const int32_t cc = on ? c : C - 1;  // lanes past C read a valid column, store nothing
        float acc[kContract ? 1 : M];
#pragma unroll
        for (int m = 0; m < (kContract ? 1 : M); ++m) acc[m] = 0.f;
        // the row's edges 64 at a time: lane l fetches the column and the basis
        // row of edge eb + l (lanes past the chunk fetch edge eb's), and the edge
        // loop reads them back lane by lane
        for (int32_t eb = e0; eb < e1; eb += 64) {
            const int32_t cnt = e1 - eb < 64 ? e1 - eb : 64;
            const int32_t ei = lane < cnt ? eb + lane : eb;
            const int32_t jl = idx[ei];
            const int64_t el = perm ? perm[ei] : ei;
            float vl[M];
#pragma unroll
            for (int m = 0; m < M; ++m) vl[m] = v[el * M + m];
            for (int32_t t0 = 0; t0 < cnt; t0 += U) {
                float x[U][kContract ? M : 1], w[U][M];
                // a slot past the chunk's end reloads edge t0 (so every load is
                // unconditional) and is then zeroed
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const bool ok = t0 + u < cnt;
                    const int32_t t = ok ? t0 + u : t0;
                    const int32_t j = __builtin_amdgcn_readlane(jl, t);
#pragma unroll
                    for (int m = 0; m < M; ++m)
                        w[u][m] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(vl[m]), t));
                    if (kContract) {
#pragma unroll
                        for (int m = 0; m < M; ++m) x[u][m] = ldx(X, ((int64_t)j * M + m) * C + cc);
                    } else {
                        x[u][0] = ldx(X, (int64_t)j * C + cc);
                    }
                    // zeroed by a mask, not a branch: a branch's join would wait
                    // for every load in flight
                    const uint32_t keep = ok ? 0xFFFFFFFFu : 0u;
#pragma unroll
                    for (int m = 0; m < M; ++m) w[u][m] = __uint_as_float(__float_as_uint(w[u][m]) & keep);
#pragma unroll
                    for (int m = 0; m < (kContract ? M : 1); ++m)
                        x[u][m] = __uint_as_float(__float_as_uint(x[u][m]) & keep);
                }
                // edges in pattern order, m ascending; a missing edge adds 0 * 0
#pragma unroll
                for (int u = 0; u < U; ++u) {
#pragma unroll
                    for (int m = 0; m < M; ++m) {
                        if (kContract) acc[0] += w[u][m] * x[u][m];
                        else acc[m] += w[u][m] * x[u][0];
                    }
                }
            }
        }
        if (on) {
            if (kContract) {
                out[(int64_t)r * C + c] = acc[0];
            } else {
#pragma unroll
                for (int m = 0; m < M; ++m) out[(int64_t)r * M * C + (int64_t)m * C + c] = acc[m];
            }
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
