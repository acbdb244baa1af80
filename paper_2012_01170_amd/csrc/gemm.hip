// Dense contractions of the convolution on the matrix cores:
//   C[R, N] = A[R, K] x B[K, N]
// with arbitrary element strides for A, B and C (so transposed operands need
// no copy), float32 or bf16 operands (bf16 is widened exactly to float32),
// float32 MFMA (v_mfma_f32_16x16x4_f32) and float32 accumulation.
//
// Tiling: a 256-thread block owns a 64 x 64 tile of C; each of its four
// waves owns a 32 x 32 quarter as 2 x 2 MFMA tiles of 16 x 16.  K advances in
// slabs of 16 staged through LDS.  Large K with few tiles is split over
// blockIdx.z; the partial tiles are summed afterwards in split order, so the
// result does not depend on scheduling.
#include "common.hpp"
#include "gemm.hpp"

namespace sbc {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kTile = 64;
constexpr int kSlab = 16;

__device__ __forceinline__ float ld(const float *p, int64_t i) { return p[i]; }
__device__ __forceinline__ float ld(const uint16_t *p, int64_t i) {
    return __uint_as_float((uint32_t)p[i] << 16);
}

template <typename AT, typename BT>
__global__ void __launch_bounds__(256)
    gemm_kernel(const AT *__restrict__ A, int64_t sa_r, int64_t sa_k, const BT *__restrict__ B,
                int64_t sb_k, int64_t sb_n, float *__restrict__ C, int64_t sc_r, int64_t sc_n,
                int32_t R, int32_t N, int64_t K, int64_t k_chunk, float *__restrict__ partial) {
    __shared__ float As[kSlab][kTile + 4];
    __shared__ float Bs[kSlab][kTile + 4];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int32_t r0 = blockIdx.y * kTile;
    const int32_t n0 = blockIdx.x * kTile;
    const int64_t kb = (int64_t)blockIdx.z * k_chunk;
    const int64_t ke = (kb + k_chunk < K) ? kb + k_chunk : K;
    const int wr = (wave >> 1) * 32;
    const int wn = (wave & 1) * 32;
    floatx4 acc[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) acc[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};

    const bool a_k_contig = sa_k == 1;
    const bool b_n_contig = sb_n == 1;
    for (int64_t k0 = kb; k0 < ke; k0 += kSlab) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int idx = tid + 256 * q;
            int rl, kl;
            if (a_k_contig) { kl = idx & 15; rl = idx >> 4; } else { rl = idx & 63; kl = idx >> 6; }
            const int32_t r = r0 + rl;
            const int64_t k = k0 + kl;
            As[kl][rl] = (r < R && k < ke) ? ld(A, (int64_t)r * sa_r + k * sa_k) : 0.f;
            int nl, kl2;
            if (b_n_contig) { nl = idx & 63; kl2 = idx >> 6; } else { kl2 = idx & 15; nl = idx >> 4; }
            const int32_t n = n0 + nl;
            const int64_t k2 = k0 + kl2;
            Bs[kl2][nl] = (n < N && k2 < ke) ? ld(B, k2 * sb_k + (int64_t)n * sb_n) : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int k4 = 0; k4 < kSlab / 4; ++k4) {
            const int kk = k4 * 4 + (lane >> 4);
            float a[2], b[2];
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                a[t] = As[kk][wr + 16 * t + (lane & 15)];
                b[t] = Bs[kk][wn + 16 * t + (lane & 15)];
            }
#pragma unroll
            for (int ta = 0; ta < 2; ++ta)
#pragma unroll
                for (int tb = 0; tb < 2; ++tb)
                    acc[ta][tb] =
                        __builtin_amdgcn_mfma_f32_16x16x4f32(a[ta], b[tb], acc[ta][tb], 0, 0, 0);
        }
        __syncthreads();
    }
    // D layout of a 16x16 MFMA tile: lane holds column (lane & 15), rows 4*(lane >> 4) + 0..3
#pragma unroll
    for (int ta = 0; ta < 2; ++ta)
#pragma unroll
        for (int tb = 0; tb < 2; ++tb)
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) {
                const int32_t row = r0 + wr + 16 * ta + 4 * (lane >> 4) + rr;
                const int32_t col = n0 + wn + 16 * tb + (lane & 15);
                if (row < R && col < N) {
                    if (partial)
                        partial[((int64_t)blockIdx.z * R + row) * N + col] = acc[ta][tb][rr];
                    else
                        C[(int64_t)row * sc_r + (int64_t)col * sc_n] = acc[ta][tb][rr];
                }
            }
}

__global__ void splitk_reduce_kernel(const float *__restrict__ partial, int32_t S, int32_t R,
                                     int32_t N, float *__restrict__ C, int64_t sc_r, int64_t sc_n) {
    const int64_t total = (int64_t)R * N;
    for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < total;
         x += (int64_t)gridDim.x * blockDim.x) {
        float s = 0.f;
        for (int32_t z = 0; z < S; ++z) s += partial[(int64_t)z * total + x];
        const int32_t row = (int32_t)(x / N), col = (int32_t)(x % N);
        C[(int64_t)row * sc_r + (int64_t)col * sc_n] = s;
    }
}

}  // namespace

int32_t gemm_splits(int32_t R, int32_t N, int64_t K) {
    const int64_t tiles = (int64_t)((R + kTile - 1) / kTile) * ((N + kTile - 1) / kTile);
    if (tiles <= 0 || K <= 0) return 1;
    int64_t s = (1024 + tiles - 1) / tiles;
    const int64_t by_k = (K + 511) / 512;  // at least 512 of K per split
    if (s > by_k) s = by_k;
    if (s > 256) s = 256;
    return s < 1 ? 1 : (int32_t)s;
}

size_t gemm_workspace_floats(int32_t R, int32_t N, int64_t K) {
    const int32_t s = gemm_splits(R, N, K);
    return s > 1 ? (size_t)s * (size_t)R * (size_t)N : 0;
}

sbc_status gemm(const void *A, bool a_bf16, int64_t sa_r, int64_t sa_k, const void *B,
                bool b_bf16, int64_t sb_k, int64_t sb_n, float *C, int64_t sc_r, int64_t sc_n,
                int32_t R, int32_t N, int64_t K, float *partial_ws, hipStream_t stream,
                const char *trace) {
    if (R <= 0 || N <= 0) return SBC_OK;
    trace_before(trace, stream);
    const int32_t S = gemm_splits(R, N, K);
    int64_t k_chunk = S > 1 ? (K + S - 1) / S : (K > 0 ? K : 1);
    k_chunk = (k_chunk + kSlab - 1) / kSlab * kSlab;
    const int32_t Sz = K > 0 ? (int32_t)((K + k_chunk - 1) / k_chunk) : 1;
    dim3 grid((N + kTile - 1) / kTile, (R + kTile - 1) / kTile, Sz);
    float *part = Sz > 1 ? partial_ws : nullptr;
#define SBC_GEMM_LAUNCH(AT, BT)                                                               \
    hipLaunchKernelGGL((gemm_kernel<AT, BT>), grid, dim3(256), 0, stream,                      \
                       static_cast<const AT *>(A), sa_r, sa_k, static_cast<const BT *>(B),     \
                       sb_k, sb_n, C, sc_r, sc_n, R, N, K, k_chunk, part)
    if (!a_bf16 && !b_bf16) SBC_GEMM_LAUNCH(float, float);
    else if (!a_bf16 && b_bf16) SBC_GEMM_LAUNCH(float, uint16_t);
    else if (a_bf16 && !b_bf16) SBC_GEMM_LAUNCH(uint16_t, float);
    else SBC_GEMM_LAUNCH(uint16_t, uint16_t);
#undef SBC_GEMM_LAUNCH
    SBC_LAUNCH_CHECK();
    if (part) {
        int64_t blocks = ((int64_t)R * N + 255) / 256;
        if (blocks > 4096) blocks = 4096;
        hipLaunchKernelGGL(splitk_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, stream,
                           part, Sz, R, N, C, sc_r, sc_n);
        SBC_LAUNCH_CHECK();
    }
    trace_after(trace, stream);
    return SBC_OK;
}

}  // namespace sbc
