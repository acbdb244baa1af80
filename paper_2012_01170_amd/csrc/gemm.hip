// Dense contractions of the convolution on the matrix cores:
//   C[R, N] = A[R, K] x B[K, N]
// with arbitrary element strides for A, B and C (so transposed operands need
// no copy), float32 or bf16 operands (bf16 is widened exactly to float32),
// float32 MFMA (v_mfma_f32_16x16x4_f32) and float32 accumulation.
//
// Tiling: a 256-thread block owns a BM x BN tile of C (128 x 128, or 64 x
// 64 when C is small and K long); its four waves own BM/2 x BN/2 quarters as
// grids of 16 x 16 MFMA tiles.  K advances in slabs of 16 (32 for the 64 x 64
// tile on vector loads) held in two LDS
// buffers: every thread loads its share of slab s+1 into registers while the
// waves multiply slab s, then stores it into the other buffer (one block
// barrier per slab).  Large K with few tiles is split over blockIdx.z; the
// partial tiles are summed afterwards in split order, so the result does not
// depend on scheduling.
#include "common.hpp"
#include "gemm.hpp"

namespace sbc {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
// K per LDS slab: 16, or kDeepSlab for the 64 x 64 tile with both operands
// on vector loads, whose short slabs would otherwise leave its few MFMAs per
// slab waiting on each slab's memory round trip (the element-wise loaders
// would spill at that depth, and the 128 x 128 tile's registers hold only
// 16).  Split-K chunks are multiples of kChunkAlign, a multiple of both.
constexpr int kDeepSlab = 32;
constexpr int kChunkAlign = 64;
template <int BT, bool kVecA, bool kVecB>
constexpr int slab_for() { return (BT == 64 && kVecA && kVecB) ? kDeepSlab : 16; }
static_assert(kChunkAlign % kDeepSlab == 0 && kChunkAlign % 16 == 0, "chunks hold whole slabs");

__device__ __forceinline__ float ld(const float *p, int64_t i) { return p[i]; }
__device__ __forceinline__ float ld(const uint16_t *p, int64_t i) {
    return __uint_as_float((uint32_t)p[i] << 16);
}

// kPer consecutive elements of a unit-stride run starting at p[off], of which
// the first `valid` exist (the rest read as 0): 16-byte loads when the run is
// whole (kVec: the caller has checked that such runs are 16-byte aligned),
// else element by element.
template <typename T, int kPer, bool kVec>
__device__ __forceinline__ void load_run(const T *__restrict__ p, int64_t off, int valid,
                                         float *out) {
    if constexpr (kVec) {
        if (valid >= kPer) {
            if constexpr (sizeof(T) == 4) {
#pragma unroll
                for (int q = 0; q < kPer; q += 4) {
                    const float4 x = *reinterpret_cast<const float4 *>(p + off + q);
                    out[q] = x.x;
                    out[q + 1] = x.y;
                    out[q + 2] = x.z;
                    out[q + 3] = x.w;
                }
            } else if constexpr (kPer % 8 == 0) {
#pragma unroll
                for (int q8 = 0; q8 < kPer; q8 += 8) {
                    const uint4 x = *reinterpret_cast<const uint4 *>(p + off + q8);
                    const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        out[q8 + 2 * q] = __uint_as_float(w[q] << 16);
                        out[q8 + 2 * q + 1] = __uint_as_float(w[q] & 0xFFFF0000u);
                    }
                }
            } else {
                static_assert(kPer == 4, "runs of 4, or of a multiple of 8, bf16 elements");
                const uint2 x = *reinterpret_cast<const uint2 *>(p + off);
                const uint32_t w[2] = {x.x, x.y};
#pragma unroll
                for (int q = 0; q < 2; ++q) {
                    out[2 * q] = __uint_as_float(w[q] << 16);
                    out[2 * q + 1] = __uint_as_float(w[q] & 0xFFFF0000u);
                }
            }
            return;
        }
    }
#pragma unroll
    for (int q = 0; q < kPer; ++q) out[q] = q < valid ? ld(p, off + q) : 0.f;
}

// One operand slab, [kSlab][BT] in LDS (BT = the tile's rows of A or columns
// of B), loaded by 256 threads, BT * kSlab / 256 elements each: runs along the
// operand's contiguous index (k, or the row / column index), so that
// neighbouring threads read neighbouring addresses.  kVec: the contiguous
// index has unit stride and its runs are 16-byte aligned (vector loads).
template <int BT, int kSlab, typename T, bool kVec>
struct SlabLoader {
    static constexpr int kPer = BT * kSlab / kThreads;  // 8 (128 x 16, 64 x 32) or 4 (64 x 16)
    float v[kPer];
    // element (t, k) of the operand at p[t * s_t + k * s_k], t < n_t, k < k_end
    __device__ __forceinline__ void load(const T *__restrict__ p, int64_t s_t, int64_t s_k,
                                         int32_t t0, int32_t n_t, int64_t k0, int64_t k_end,
                                         bool k_contig) {
        const int tid = threadIdx.x;
        if (kVec && k_contig) {  // a thread takes kPer consecutive k of one row
            const int tl = tid / (kSlab / kPer);
            const int kl = (tid % (kSlab / kPer)) * kPer;
            const int32_t t = t0 + tl;
            const int64_t k = k0 + kl;
            const int64_t left = k_end - k;
            const int valid = t < n_t ? (left >= kPer ? kPer : (left > 0 ? (int)left : 0)) : 0;
            load_run<T, kPer, kVec>(p, (int64_t)t * s_t + k, valid, v);
            return;
        }
        if (kVec) {              // a thread takes kPer consecutive rows at one k
            const int kl = tid / (BT / kPer);
            const int tl = (tid % (BT / kPer)) * kPer;
            const int32_t t = t0 + tl;
            const int64_t k = k0 + kl;
            const int32_t left = n_t - t;
            const int valid = k < k_end ? (left >= kPer ? kPer : (left > 0 ? left : 0)) : 0;
            load_run<T, kPer, kVec>(p, (int64_t)t + k * s_k, valid, v);
            return;
        }
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            int tl, kl;
            if (k_contig) {  // a thread takes kPer consecutive k of one row
                tl = tid / (kSlab / kPer);
                kl = (tid % (kSlab / kPer)) * kPer + q;
            } else {         // a thread takes kPer consecutive rows at one k
                kl = tid / (BT / kPer);
                tl = (tid % (BT / kPer)) * kPer + q;
            }
            const int32_t t = t0 + tl;
            const int64_t k = k0 + kl;
            v[q] = (t < n_t && k < k_end) ? ld(p, (int64_t)t * s_t + k * s_k) : 0.f;
        }
    }
    __device__ __forceinline__ void store(float (*S)[BT + 4], bool k_contig) const {
        const int tid = threadIdx.x;
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            int tl, kl;
            if (k_contig) {
                tl = tid / (kSlab / kPer);
                kl = (tid % (kSlab / kPer)) * kPer + q;
            } else {
                kl = tid / (BT / kPer);
                tl = (tid % (BT / kPer)) * kPer + q;
            }
            S[kl][tl] = v[q];
        }
    }
};

template <int BM, int BN, typename AT, typename BT, bool kVecA, bool kVecB>
__global__ void __launch_bounds__(kThreads, 2)
    gemm_kernel(const AT *__restrict__ A, int64_t sa_r, int64_t sa_k, const BT *__restrict__ B,
                int64_t sb_k, int64_t sb_n, float *__restrict__ C, int64_t sc_r, int64_t sc_n,
                int32_t R, int32_t N, int64_t K, int64_t k_chunk, float *__restrict__ partial) {
    constexpr int TM = BM / 32, TN = BN / 32;  // 16x16 tiles per wave (2 x 2 waves)
    static_assert(BM == BN, "square tiles");
    constexpr int kSlab = slab_for<BM, kVecA, kVecB>();
    __shared__ float As[2][kSlab][BM + 4];
    __shared__ float Bs[2][kSlab][BN + 4];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int32_t r0 = blockIdx.y * BM;
    const int32_t n0 = blockIdx.x * BN;
    const int64_t kb = (int64_t)blockIdx.z * k_chunk;
    const int64_t ke = (kb + k_chunk < K) ? kb + k_chunk : K;
    const int wr = (wave >> 1) * (BM / 2);
    const int wn = (wave & 1) * (BN / 2);
    const bool a_kc = sa_k == 1, b_kc = sb_k == 1;
    floatx4 acc[TM][TN];
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b) acc[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};

    SlabLoader<BM, kSlab, AT, kVecA> la;
    SlabLoader<BN, kSlab, BT, kVecB> lb;
    la.load(A, sa_r, sa_k, r0, R, kb, ke, a_kc);
    lb.load(B, sb_n, sb_k, n0, N, kb, ke, b_kc);
    la.store(As[0], a_kc);
    lb.store(Bs[0], b_kc);
    __syncthreads();
    int buf = 0;
    for (int64_t k0 = kb; k0 < ke; k0 += kSlab) {
        const bool more = k0 + kSlab < ke;
        if (more) {
            la.load(A, sa_r, sa_k, r0, R, k0 + kSlab, ke, a_kc);
            lb.load(B, sb_n, sb_k, n0, N, k0 + kSlab, ke, b_kc);
        }
#pragma unroll
        for (int k4 = 0; k4 < kSlab / 4; ++k4) {
            const int kk = k4 * 4 + (lane >> 4);
            float a[TM], b[TN];
#pragma unroll
            for (int t = 0; t < TM; ++t) a[t] = As[buf][kk][wr + 16 * t + (lane & 15)];
#pragma unroll
            for (int t = 0; t < TN; ++t) b[t] = Bs[buf][kk][wn + 16 * t + (lane & 15)];
#pragma unroll
            for (int ta = 0; ta < TM; ++ta)
#pragma unroll
                for (int tb = 0; tb < TN; ++tb)
                    acc[ta][tb] =
                        __builtin_amdgcn_mfma_f32_16x16x4f32(a[ta], b[tb], acc[ta][tb], 0, 0, 0);
        }
        if (more) {
            la.store(As[buf ^ 1], a_kc);
            lb.store(Bs[buf ^ 1], b_kc);
        }
        __syncthreads();
        buf ^= 1;
    }
    // D layout of a 16x16 MFMA tile: lane holds column (lane & 15), rows 4*(lane >> 4) + 0..3
#pragma unroll
    for (int ta = 0; ta < TM; ++ta)
#pragma unroll
        for (int tb = 0; tb < TN; ++tb)
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
        // split order, eight partial loads in flight
        float s = 0.f;
        for (int32_t z0 = 0; z0 < S; z0 += 8) {
            float v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j)
                v[j] = z0 + j < S ? partial[(int64_t)(z0 + j) * total + x] : 0.f;
#pragma unroll
            for (int j = 0; j < 8; ++j) s += v[j];
        }
        const int32_t row = (int32_t)(x / N), col = (int32_t)(x % N);
        C[(int64_t)row * sc_r + (int64_t)col * sc_n] = s;
    }
}

}  // namespace

// Tile of a shape: 128 x 128, or 64 x 64 when C has fewer than 128 rows or
// columns (a 128 tile would be half empty) or when the 128 tiles would give
// fewer than two blocks per CU (the 64 x 64 tiles then keep four per CU
// busy: C of 8192 x 512 with K = 128, 24.5 -> 21.6 us).
static int tile_for(int32_t R, int32_t N) {
    if (R < 128 || N < 128) return 64;
    const int64_t big = (int64_t)((R + 127) / 128) * ((N + 127) / 128);
    return big >= 512 ? 128 : 64;
}

int32_t gemm_splits(int32_t R, int32_t N, int64_t K) {
    const int t = tile_for(R, N);
    const int64_t tiles = (int64_t)((R + t - 1) / t) * ((N + t - 1) / t);
    if (tiles <= 0 || K <= 0) return 1;
    int64_t s = (512 + tiles - 1) / tiles;        // about two blocks per CU
    const int64_t by_k = (K + 127) / 128;         // at least 128 of K per split
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
    k_chunk = (k_chunk + kChunkAlign - 1) / kChunkAlign * kChunkAlign;
    const int32_t Sz = K > 0 ? (int32_t)((K + k_chunk - 1) / k_chunk) : 1;
    const int t = tile_for(R, N);
    dim3 grid((N + t - 1) / t, (R + t - 1) / t, Sz);
    float *part = Sz > 1 ? partial_ws : nullptr;
    // vector loads along an operand's unit-stride index when its runs are
    // 16-byte aligned: the base and the other stride a multiple of 16 bytes
    auto vec_ok = [](const void *p, bool bf, int64_t s_t, int64_t s_k) {
        const int64_t ve = bf ? 8 : 4;  // elements per 16 bytes
        if (reinterpret_cast<uintptr_t>(p) % 16 != 0) return false;
        if (s_k == 1) return s_t % ve == 0;
        if (s_t == 1) return s_k % ve == 0;
        return false;
    };
    const bool va = vec_ok(A, a_bf16, sa_r, sa_k), vb = vec_ok(B, b_bf16, sb_n, sb_k);
#define SBC_GEMM_LAUNCH1(TT, AT, BT, VA, VB)                                                  \
    hipLaunchKernelGGL((gemm_kernel<TT, TT, AT, BT, VA, VB>), grid, dim3(kThreads), 0, stream, \
                       static_cast<const AT *>(A), sa_r, sa_k, static_cast<const BT *>(B),     \
                       sb_k, sb_n, C, sc_r, sc_n, R, N, K, k_chunk, part)
#define SBC_GEMM_LAUNCH(TT, AT, BT)                                                           \
    if (va && vb) SBC_GEMM_LAUNCH1(TT, AT, BT, true, true);                                   \
    else if (va) SBC_GEMM_LAUNCH1(TT, AT, BT, true, false);                                   \
    else if (vb) SBC_GEMM_LAUNCH1(TT, AT, BT, false, true);                                   \
    else SBC_GEMM_LAUNCH1(TT, AT, BT, false, false)
#define SBC_GEMM_TYPES(TT)                                                                    \
    if (!a_bf16 && !b_bf16) SBC_GEMM_LAUNCH(TT, float, float);                                \
    else if (!a_bf16 && b_bf16) SBC_GEMM_LAUNCH(TT, float, uint16_t);                         \
    else if (a_bf16 && !b_bf16) SBC_GEMM_LAUNCH(TT, uint16_t, float);                         \
    else SBC_GEMM_LAUNCH(TT, uint16_t, uint16_t);
    if (t == 128) {
        SBC_GEMM_TYPES(128)
    } else {
        SBC_GEMM_TYPES(64)
    }
#undef SBC_GEMM_TYPES
#undef SBC_GEMM_LAUNCH
#undef SBC_GEMM_LAUNCH1
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
