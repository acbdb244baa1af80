// Fused kernels of the sparse basis convolution (Section 3.1: Y = sum_m
// N^(m) F W^(m), evaluated as (N F) W; its backward as the transposed
// products).  The basis values are evaluated inside the kernels from the
// coordinates (the paper computes them on the accelerator from the neighbour
// indices), or read from a materialised [E, M] array.
//
// Forward, one block per tile of TR output rows:
//   gather   G[r, m*C_in + c] = sum_e v[e, m] F[j(e), c] into LDS.  A wave
//            handles its rows in batches: the batch's edges are staged 64 at a
//            time (index and basis values, one edge per lane) in LDS, then
//            every row of the batch is owned by LPR lanes that accumulate
//            M x VEC values while walking the row's edges, loading VEC
//            contiguous channels of F[j] per edge (16-byte loads);
//   contract Y_tile = G_tile W on the matrix cores (float32: 16x16x4 f32
//            MFMA with W read from L2; bf16: G rounded to bf16 in LDS and
//            16x16x32 bf16 MFMA against a [C_out, M*C_in] copy of W).
// Backward (D-route), persistent blocks over tiles of TR input rows:
//   gather   D[j, m*C_out + p] = sum_{e=(i,j)} v[e, m] dY[i, p] through the
//            transposed pattern, into LDS (F's tile rows are staged too);
//   dF       dF_tile = D_tile Wt (Wt[(m, p), c] = W[m, c, p]) on MFMA;
//   dW       every block accumulates F_tile^T D_tile over its tiles in
//            registers; the per-block partials are summed afterwards in
//            block order, so dW does not depend on scheduling.
// Sums over edges run in pattern order inside a lane; no floating-point
// atomics are used anywhere.
#include <type_traits>

#include "basis.hpp"
#include "common.hpp"
#include "fused.hpp"

namespace sbc {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
    __builtin_amdgcn_wave_barrier();
}

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// float32 -> bf16 bits, round to nearest even (finite inputs)
__device__ __forceinline__ uint16_t f2bf(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// ---------------------------------------------------------------- basis per edge
// kBasis: 0 = read v[ev, :], SBC_BASIS_MONO4 + 1, SBC_BASIS_MONO8 + 1, SBC_BASIS_EVENT8 + 1
// (i = output index, j = input index of the edge, ev = its CSR position).
template <int M, int kBasis>
__device__ __forceinline__ void edge_basis(const sbc_geometry &g, const float *__restrict__ v,
                                           int32_t i, int32_t j, int64_t ev, double inv_r,
                                           float inv_tau, float *out) {
    if constexpr (kBasis == 0) {
#pragma unroll
        for (int m = 0; m < M; ++m) out[m] = v[ev * M + m];
    } else if constexpr (kBasis == SBC_BASIS_EVENT8 + 1) {
        const int k = event_index(g.px[i] - g.px[j], g.py[i] - g.py[j]);
        const float d = event_decay(g.t[i], g.t[j], inv_tau);
#pragma unroll
        for (int m = 0; m < M; ++m) out[m] = (m == k) ? d : 0.f;
    } else {
        point_basis<M>(g.x_out[3 * (int64_t)i], g.x_out[3 * (int64_t)i + 1],
                       g.x_out[3 * (int64_t)i + 2], g.x_in[3 * (int64_t)j],
                       g.x_in[3 * (int64_t)j + 1], g.x_in[3 * (int64_t)j + 2], inv_r, out);
    }
}

// Per-wave LDS stage of up to 64 edges: neighbour index and basis values,
// plus the row bounds of the wave's rows.
template <int M>
struct EdgeStage {
    int32_t nb[64];
    float v[64][M + 1];
    int32_t bounds[17];
};

// VEC contiguous channels of row `r` of X (float32 or bf16) as float32.
template <int C, int VEC, bool kXbf>
__device__ __forceinline__ void load_row_vec(const void *__restrict__ Xv, int32_t r, int cg,
                                             float *f) {
    if constexpr (kXbf) {
        const uint4 raw = *reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(Xv) +
                                                           (int64_t)r * C + cg * VEC);
        const uint32_t w4[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            f[2 * k] = __uint_as_float(w4[k] << 16);
            f[2 * k + 1] = __uint_as_float(w4[k] & 0xFFFF0000u);
        }
    } else {
        const float4 raw = *reinterpret_cast<const float4 *>(static_cast<const float *>(Xv) +
                                                             (int64_t)r * C + cg * VEC);
        f[0] = raw.x;
        f[1] = raw.y;
        f[2] = raw.z;
        f[3] = raw.w;
    }
}

// Gather of one wave's RPW consecutive rows into an LDS tile.
//   kT: the pattern is transposed (rows are inputs j, idx gives outputs i).
//   X [*, C] features gathered along the pattern; out tile row stride S
//   (elements), row r_local at out + r_local * S, column m*C + c.
// The wave's edges are staged 64 at a time; the rows are owned by groups of
// LPR lanes (RPB rows at once, NB rounds, all accumulators live across the
// staging chunks), and each group loads the features of 4 edges at once.
template <int M, int C, int kBasis, bool kXbf, bool kOutBf, bool kT, int RPW>
__device__ __forceinline__ void gather_rows(int32_t row_begin, int32_t n_rows,
                                            const int32_t *__restrict__ ptr,
                                            const int32_t *__restrict__ idx,
                                            const int32_t *__restrict__ perm,
                                            const float *__restrict__ v, const sbc_geometry &g,
                                            const void *__restrict__ Xv, void *out_tile, int S,
                                            int local_row0, EdgeStage<M> &st, double inv_r,
                                            float inv_tau) {
    constexpr int VEC = kXbf ? 8 : 4;
    static_assert(C % VEC == 0, "channels must be a multiple of the vector width");
    constexpr int LPR = C / VEC;                   // lanes per row
    static_assert(LPR <= 64 && 64 % LPR == 0, "row must fit a wave");
    static_assert(RPW <= 16, "row bounds stage holds 17 entries");
    constexpr int RPB_ = 64 / LPR;
    constexpr int RPB = RPB_ < RPW ? RPB_ : RPW;   // rows in flight at once
    constexpr int NB = (RPW + RPB - 1) / RPB;      // rounds over the wave's rows
    constexpr int U = 4;                           // edges loaded together
    const int lane = threadIdx.x & 63;
    const int slot = lane / LPR;
    const int cg = lane % LPR;

    if (lane <= RPW) {
        int32_t r = row_begin + lane;
        r = r < n_rows ? r : n_rows;
        r = r > 0 ? r : 0;
        st.bounds[lane] = ptr[r];
    }
    wave_lds_sync();
    const int32_t wb = st.bounds[0], we = st.bounds[RPW];
    int32_t rs[NB], re[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        const int lr = b * RPB + slot;
        const bool own = slot < RPB && lr < RPW;
        rs[b] = own ? st.bounds[lr] : 0;
        re[b] = own ? st.bounds[lr + 1] : 0;
    }
    float acc[NB][M][VEC];
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int m = 0; m < M; ++m)
#pragma unroll
            for (int k = 0; k < VEC; ++k) acc[b][m][k] = 0.f;

#pragma unroll 1
    for (int32_t c0 = wb; c0 < we; c0 += 64) {
        const int32_t e = c0 + lane;
        if (e < we) {
            int s = 0;
#pragma unroll
            for (int q = 1; q < RPW; ++q)
                if (st.bounds[q] <= e) s = q;
            const int32_t row = row_begin + s;
            const int32_t other = idx[e];
            const int64_t ev = (kBasis == 0) ? (perm ? (int64_t)perm[e] : (int64_t)e) : 0;
            float bv[M];
            if (kT)
                edge_basis<M, kBasis>(g, v, other, row, ev, inv_r, inv_tau, bv);
            else
                edge_basis<M, kBasis>(g, v, row, other, ev, inv_r, inv_tau, bv);
            st.nb[lane] = other;
#pragma unroll
            for (int m = 0; m < M; ++m) st.v[lane][m] = bv[m];
        }
        wave_lds_sync();
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            const int32_t lo = rs[b] > c0 ? rs[b] : c0;
            const int32_t hi = re[b] < c0 + 64 ? re[b] : c0 + 64;
#pragma unroll 1
            for (int32_t e2 = lo; e2 < hi; e2 += U) {
                float f[U][VEC];
                int q[U];
                bool ok[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    ok[u] = e2 + u < hi;
                    q[u] = (ok[u] ? e2 + u : lo) - c0;
                    load_row_vec<C, VEC, kXbf>(Xv, st.nb[q[u]], cg, f[u]);
                }
#pragma unroll
                for (int u = 0; u < U; ++u) {
#pragma unroll
                    for (int m = 0; m < M; ++m) {
                        const float vm = ok[u] ? st.v[q[u]][m] : 0.f;
#pragma unroll
                        for (int k = 0; k < VEC; ++k) acc[b][m][k] += vm * f[u][k];
                    }
                }
            }
        }
        wave_lds_sync();
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        const int lr = b * RPB + slot;
        if (slot < RPB && lr < RPW) {
#pragma unroll
            for (int m = 0; m < M; ++m) {
                if constexpr (kOutBf) {
                    uint16_t *o = static_cast<uint16_t *>(out_tile) +
                                  (int64_t)(local_row0 + lr) * S + m * C + cg * VEC;
#pragma unroll
                    for (int k = 0; k < VEC; ++k) o[k] = f2bf(acc[b][m][k]);
                } else {
                    float *o = static_cast<float *>(out_tile) + (int64_t)(local_row0 + lr) * S +
                               m * C + cg * VEC;
#pragma unroll
                    for (int k = 0; k < VEC; ++k) o[k] = acc[b][m][k];
                }
            }
        }
    }
}

// acc[u][t] += A_tile[16 rb_u .., :] x B[:, 16 cb_t ..] for the 16x16 blocks of
// one wave (rb_u = wr + NRG u, cb_t = wc + NCBW t).  A sits in LDS (row stride
// S elements), B [K, NCOL] in global memory (float32) or, for bf16, as
// B^T [NCOL, K]; the B fragments of the next k-group are loaded while the
// current group is multiplied.
template <int K, int NCOL, int S, int WRB, int WCB, int NCBW, int NRG>
__device__ __forceinline__ void mfma_lds_x_global_f32(const float *As, const float *__restrict__ B,
                                                      int wr, int wc,
                                                      floatx4 (&acc)[WRB][WCB]) {
    constexpr int KG = 32;  // 8 MFMA k-steps of 4
    static_assert(K % KG == 0, "K must be a multiple of 32");
    const int lane = threadIdx.x & 63;
    const int lr = lane >> 4, lc = lane & 15;
    float bc[8][WCB], bn[8][WCB];
#pragma unroll
    for (int s = 0; s < 8; ++s)
#pragma unroll
        for (int t = 0; t < WCB; ++t) bc[s][t] = B[(4 * s + lr) * NCOL + 16 * (wc + NCBW * t) + lc];
#pragma unroll 1
    for (int k0 = 0; k0 < K; k0 += KG) {
        const int kn = k0 + KG < K ? k0 + KG : k0;
#pragma unroll
        for (int s = 0; s < 8; ++s)
#pragma unroll
            for (int t = 0; t < WCB; ++t)
                bn[s][t] = B[(kn + 4 * s + lr) * NCOL + 16 * (wc + NCBW * t) + lc];
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            float a[WRB];
#pragma unroll
            for (int u = 0; u < WRB; ++u) a[u] = As[(16 * (wr + NRG * u) + lc) * S + k0 + 4 * s + lr];
#pragma unroll
            for (int u = 0; u < WRB; ++u)
#pragma unroll
                for (int t = 0; t < WCB; ++t)
                    acc[u][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[u], bc[s][t], acc[u][t], 0, 0, 0);
        }
#pragma unroll
        for (int s = 0; s < 8; ++s)
#pragma unroll
            for (int t = 0; t < WCB; ++t) bc[s][t] = bn[s][t];
    }
}

template <int K, int S, int WRB, int WCB, int NCBW, int NRG>
__device__ __forceinline__ void mfma_lds_x_global_bf16(const uint16_t *As,
                                                       const uint16_t *__restrict__ Bt, int wr,
                                                       int wc, floatx4 (&acc)[WRB][WCB]) {
    constexpr int KG = 128;  // 4 MFMA k-steps of 32
    static_assert(K % KG == 0, "K must be a multiple of 128");
    const int lane = threadIdx.x & 63;
    const int lk = 8 * (lane >> 4), lc = lane & 15;
    bf16x8 bc[4][WCB], bn[4][WCB];
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int t = 0; t < WCB; ++t)
            bc[s][t] = *reinterpret_cast<const bf16x8 *>(
                Bt + (int64_t)(16 * (wc + NCBW * t) + lc) * K + 32 * s + lk);
#pragma unroll 1
    for (int k0 = 0; k0 < K; k0 += KG) {
        const int kn = k0 + KG < K ? k0 + KG : k0;
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int t = 0; t < WCB; ++t)
                bn[s][t] = *reinterpret_cast<const bf16x8 *>(
                    Bt + (int64_t)(16 * (wc + NCBW * t) + lc) * K + kn + 32 * s + lk);
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            bf16x8 a[WRB];
#pragma unroll
            for (int u = 0; u < WRB; ++u)
                a[u] = *reinterpret_cast<const bf16x8 *>(
                    &As[(16 * (wr + NRG * u) + lc) * S + k0 + 32 * s + lk]);
#pragma unroll
            for (int u = 0; u < WRB; ++u)
#pragma unroll
                for (int t = 0; t < WCB; ++t)
                    acc[u][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[u], bc[s][t], acc[u][t], 0, 0, 0);
        }
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int t = 0; t < WCB; ++t) bc[s][t] = bn[s][t];
    }
}

// Tile rows per block: keep the float32 G tile within 64 KiB (two blocks per CU).
template <int K, bool kBf>
constexpr int tile_rows() {
    return (K * (kBf ? 2 : 4) * 64 <= 65536) ? 64 : 32;
}

// ================================================================ forward
template <int M, int CI, int CO, int kBasis, bool kBf>
__global__ void __launch_bounds__(256, 2)
    fwd_fused_kernel(int32_t n_out, const int32_t *__restrict__ row_ptr,
                     const int32_t *__restrict__ col_idx, const float *__restrict__ v,
                     sbc_geometry g, const void *__restrict__ F, const void *__restrict__ Wop,
                     float *__restrict__ Y) {
    constexpr int K = M * CI;
    constexpr int TR = tile_rows<K, kBf>();
    constexpr int S = K + (kBf ? 8 : 4);           // padded LDS row (elements)
    constexpr int NRB = TR / 16, NCB = CO / 16;
    static_assert(CO % 16 == 0 && CI % 4 == 0, "shape");
    constexpr int NCBW = NCB < 4 ? NCB : 4;        // column groups of waves
    constexpr int NRG = 4 / NCBW;                  // row groups of waves
    static_assert(NCB % NCBW == 0 && NRB % NRG == 0, "tile split");
    constexpr int WCB = NCB / NCBW, WRB = NRB / NRG;

    using GT = typename std::conditional<kBf, uint16_t, float>::type;
    __shared__ __attribute__((aligned(16))) GT Gs[TR * S];
    __shared__ EdgeStage<M> stage[4];

    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const int32_t row0 = blockIdx.x * TR;
    const double inv_r = 1.0 / (double)g.radius;
    const float inv_tau = 1.0f / g.tau;

    gather_rows<M, CI, kBasis, kBf, kBf, false, TR / 4>(row0 + w * (TR / 4), n_out, row_ptr,
                                                         col_idx, nullptr, v, g, F, Gs, S,
                                                         w * (TR / 4), stage[w], inv_r, inv_tau);
    __syncthreads();

    const int wc = w % NCBW, wr = w / NCBW;
    floatx4 acc[WRB][WCB];
#pragma unroll
    for (int u = 0; u < WRB; ++u)
#pragma unroll
        for (int t = 0; t < WCB; ++t) acc[u][t] = floatx4{0.f, 0.f, 0.f, 0.f};

    if constexpr (!kBf)
        mfma_lds_x_global_f32<K, CO, S, WRB, WCB, NCBW, NRG>(
            Gs, static_cast<const float *>(Wop), wr, wc, acc);
    else
        mfma_lds_x_global_bf16<K, S, WRB, WCB, NCBW, NRG>(
            Gs, static_cast<const uint16_t *>(Wop), wr, wc, acc);
#pragma unroll
    for (int u = 0; u < WRB; ++u)
#pragma unroll
        for (int t = 0; t < WCB; ++t)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int32_t row = row0 + 16 * (wr + NRG * u) + 4 * (lane >> 4) + r;
                if (row < n_out) Y[(int64_t)row * CO + 16 * (wc + NCBW * t) + (lane & 15)] = acc[u][t][r];
            }
}

// ================================================================ backward (D-route)
template <int K2, bool kBf>
constexpr int bwd_tile_rows() {
    return (K2 * (kBf ? 2 : 4) * 64 <= 65536) ? 64 : 32;
}

template <int M, int CI, int CO, int kBasis, bool kBf>
__global__ void __launch_bounds__(256, 1)
    bwd_fused_kernel(int32_t n_in, int32_t n_tiles, const int32_t *__restrict__ col_ptr,
                     const int32_t *__restrict__ row_idx, const int32_t *__restrict__ perm,
                     const float *__restrict__ v, sbc_geometry g, const void *__restrict__ Fv,
                     const void *__restrict__ dY, const void *__restrict__ Wop,
                     float *__restrict__ dF, float *__restrict__ dW_part) {
    // dF == nullptr: no input gradient; dW_part == nullptr: no weight gradient
    constexpr int K2 = M * CO;
    constexpr int TR = bwd_tile_rows<K2, kBf>();
    constexpr int SD = K2 + (kBf ? 8 : 4);
    constexpr int SF = CI + 4;
    static_assert(CI % 16 == 0 && CO % 16 == 0, "shape");
    // dF tile [TR, CI]: 16x16 blocks over waves
    constexpr int NRB = TR / 16, NCB = CI / 16;
    constexpr int NCBW = NCB < 4 ? NCB : 4;
    constexpr int NRG = 4 / NCBW;
    static_assert(NCB % NCBW == 0 && NRB % NRG == 0, "dF split");
    constexpr int WCB = NCB / NCBW, WRB = NRB / NRG;
    // dW [CI, K2]: each wave owns K2/4 columns, all CI rows
    constexpr int NWB = (K2 / 16) / 4;                 // column blocks per wave
    constexpr int NIB = CI / 16;                       // row blocks
    static_assert((K2 / 16) % 4 == 0, "dW split");

    using DT = typename std::conditional<kBf, uint16_t, float>::type;
    __shared__ __attribute__((aligned(16))) DT Ds[TR * SD];
    __shared__ __attribute__((aligned(16))) float Fs[TR * SF];
    __shared__ EdgeStage<M> stage[4];

    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const double inv_r = 1.0 / (double)g.radius;
    const float inv_tau = 1.0f / g.tau;
    const int wc = w % NCBW, wr = w / NCBW;

    floatx4 accw[NIB][NWB];
#pragma unroll
    for (int a = 0; a < NIB; ++a)
#pragma unroll
        for (int b = 0; b < NWB; ++b) accw[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};

#pragma unroll 1
    for (int32_t tile = blockIdx.x; tile < n_tiles; tile += gridDim.x) {
        const int32_t row0 = tile * TR;
        // F rows of the tile -> Fs (float32), zero past n_in
        for (int x = threadIdx.x; x < TR * CI; x += 256) {
            const int r = x / CI, c = x % CI;
            const int32_t row = row0 + r;
            float f = 0.f;
            if (row < n_in) {
                if constexpr (kBf)
                    f = bf2f(static_cast<const uint16_t *>(Fv)[(int64_t)row * CI + c]);
                else
                    f = static_cast<const float *>(Fv)[(int64_t)row * CI + c];
            }
            Fs[r * SF + c] = f;
        }
        gather_rows<M, CO, kBasis, kBf, kBf, true, TR / 4>(row0 + w * (TR / 4), n_in, col_ptr,
                                                            row_idx, perm, v, g, dY, Ds, SD,
                                                            w * (TR / 4), stage[w], inv_r,
                                                            inv_tau);
        __syncthreads();

        // ---- dF_tile = D_tile Wt  ([TR, K2] x [K2, CI])
        if (dF) {
        floatx4 acc[WRB][WCB];
#pragma unroll
        for (int u = 0; u < WRB; ++u)
#pragma unroll
            for (int t = 0; t < WCB; ++t) acc[u][t] = floatx4{0.f, 0.f, 0.f, 0.f};
        if constexpr (!kBf)
            mfma_lds_x_global_f32<K2, CI, SD, WRB, WCB, NCBW, NRG>(
                Ds, static_cast<const float *>(Wop), wr, wc, acc);
        else
            mfma_lds_x_global_bf16<K2, SD, WRB, WCB, NCBW, NRG>(
                Ds, static_cast<const uint16_t *>(Wop), wr, wc, acc);
#pragma unroll
        for (int u = 0; u < WRB; ++u)
#pragma unroll
            for (int t = 0; t < WCB; ++t)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int32_t row = row0 + 16 * (wr + NRG * u) + 4 * (lane >> 4) + r;
                    if (row < n_in)
                        dF[(int64_t)row * CI + 16 * (wc + NCBW * t) + (lane & 15)] = acc[u][t][r];
                }
        }

        // ---- dW += F_tile^T D_tile  ([CI, TR] x [TR, K2]), float32 MFMA over the tile rows
        if (dW_part) {
#pragma unroll 2
        for (int k0 = 0; k0 < TR; k0 += 4) {
            const int kk = k0 + (lane >> 4);
            float a[NIB];
#pragma unroll
            for (int ib = 0; ib < NIB; ++ib) a[ib] = Fs[kk * SF + 16 * ib + (lane & 15)];
#pragma unroll
            for (int nb = 0; nb < NWB; ++nb) {
                const int col = 16 * (w * NWB + nb) + (lane & 15);
                float bb;
                if constexpr (kBf)
                    bb = bf2f(Ds[kk * SD + col]);
                else
                    bb = Ds[kk * SD + col];
#pragma unroll
                for (int ib = 0; ib < NIB; ++ib)
                    accw[ib][nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[ib], bb, accw[ib][nb], 0, 0, 0);
            }
        }
        }
        __syncthreads();
    }
    if (!dW_part) return;
    // this block's partial dW, layout [CI, K2]
    float *out = dW_part + (int64_t)blockIdx.x * CI * K2;
#pragma unroll
    for (int ib = 0; ib < NIB; ++ib)
#pragma unroll
        for (int nb = 0; nb < NWB; ++nb)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                out[(16 * ib + 4 * (lane >> 4) + r) * K2 + 16 * (w * NWB + nb) + (lane & 15)] =
                    accw[ib][nb][r];
}

// dW[m, c, p] = sum_b part[b, c, m*CO + p].  A block of 256 threads owns 32
// consecutive partial positions; its 8 thread groups each sum a fixed,
// contiguous range of blocks in order, and the 8 group sums are then added in
// group order, so the result is independent of scheduling.
constexpr int kReduceGroups = 8;

__global__ void __launch_bounds__(256)
    dw_reduce_kernel(const float *__restrict__ part, int32_t n_parts, int32_t M, int32_t CI,
                     int32_t CO, float *__restrict__ dW) {
    __shared__ float sums[kReduceGroups][32];
    const int64_t K2 = (int64_t)M * CO;
    const int64_t total = (int64_t)CI * K2;
    const int g = threadIdx.x >> 5;
    const int64_t off = (int64_t)blockIdx.x * 32 + (threadIdx.x & 31);
    const int32_t per = (n_parts + kReduceGroups - 1) / kReduceGroups;
    const int32_t b0 = g * per;
    const int32_t b1 = b0 + per < n_parts ? b0 + per : n_parts;
    float s = 0.f;
    if (off < total)
        for (int32_t b = b0; b < b1; ++b) s += part[(int64_t)b * total + off];
    sums[g][threadIdx.x & 31] = s;
    __syncthreads();
    if (g == 0 && off < total) {
        float t = 0.f;
#pragma unroll
        for (int q = 0; q < kReduceGroups; ++q) t += sums[q][threadIdx.x & 31];
        // off = c*K2 + m*CO + p  ->  dW[(m*CI + c)*CO + p]
        const int64_t c = off / K2, mp = off % K2;
        const int64_t m = mp / CO, p = mp % CO;
        dW[(m * CI + c) * CO + p] = t;
    }
}

// W [M, CI, CO] (float32 or bf16) -> bf16 copy with element (m, c, p) at m*s_m + c*s_c + p*s_p
template <typename T>
__global__ void w_to_bf16_kernel(const T *__restrict__ W, int32_t M, int32_t CI, int32_t CO,
                                 int64_t s_m, int64_t s_c, int64_t s_p, uint16_t *__restrict__ out) {
    const int64_t total = (int64_t)M * CI * CO;
    for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < total;
         x += (int64_t)gridDim.x * blockDim.x) {
        const int32_t p = (int32_t)(x % CO);
        const int32_t c = (int32_t)((x / CO) % CI);
        const int32_t m = (int32_t)(x / ((int64_t)CO * CI));
        uint16_t b;
        if constexpr (sizeof(T) == 2) b = W[x]; else b = f2bf(W[x]);
        out[m * s_m + c * s_c + p * s_p] = b;
    }
}

// W [M, CI, CO] float32 -> float32 copy with element (m, c, p) at m*s_m + c*s_c + p*s_p
__global__ void w_perm_f32_kernel(const float *__restrict__ W, int32_t M, int32_t CI, int32_t CO,
                                  int64_t s_m, int64_t s_c, int64_t s_p, float *__restrict__ out) {
    const int64_t total = (int64_t)M * CI * CO;
    for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < total;
         x += (int64_t)gridDim.x * blockDim.x) {
        const int32_t p = (int32_t)(x % CO);
        const int32_t c = (int32_t)((x / CO) % CI);
        const int32_t m = (int32_t)(x / ((int64_t)CO * CI));
        out[m * s_m + c * s_c + p * s_p] = W[x];
    }
}

// ---------------------------------------------------------------- dispatch tables
using FwdFn = void (*)(int32_t, const int32_t *, const int32_t *, const float *, sbc_geometry,
                       const void *, const void *, float *);
using BwdFn = void (*)(int32_t, int32_t, const int32_t *, const int32_t *, const int32_t *,
                       const float *, sbc_geometry, const void *, const void *, const void *,
                       float *, float *);

struct Shape {
    int M, CI, CO;
    bool bf;
};

template <int M, int CI, int CO, bool kBf>
FwdFn fwd_for(int basis_mode) {
    switch (basis_mode) {
        case 0: return fwd_fused_kernel<M, CI, CO, 0, kBf>;
        case SBC_BASIS_MONO4 + 1:
            if constexpr (M == 4) return fwd_fused_kernel<M, CI, CO, SBC_BASIS_MONO4 + 1, kBf>;
            return nullptr;
        case SBC_BASIS_MONO8 + 1:
            if constexpr (M == 8) return fwd_fused_kernel<M, CI, CO, SBC_BASIS_MONO8 + 1, kBf>;
            return nullptr;
        case SBC_BASIS_EVENT8 + 1:
            if constexpr (M == 8) return fwd_fused_kernel<M, CI, CO, SBC_BASIS_EVENT8 + 1, kBf>;
            return nullptr;
    }
    return nullptr;
}

template <int M, int CI, int CO, bool kBf>
BwdFn bwd_for(int basis_mode) {
    switch (basis_mode) {
        case 0: return bwd_fused_kernel<M, CI, CO, 0, kBf>;
        case SBC_BASIS_MONO4 + 1:
            if constexpr (M == 4) return bwd_fused_kernel<M, CI, CO, SBC_BASIS_MONO4 + 1, kBf>;
            return nullptr;
        case SBC_BASIS_MONO8 + 1:
            if constexpr (M == 8) return bwd_fused_kernel<M, CI, CO, SBC_BASIS_MONO8 + 1, kBf>;
            return nullptr;
        case SBC_BASIS_EVENT8 + 1:
            if constexpr (M == 8) return bwd_fused_kernel<M, CI, CO, SBC_BASIS_EVENT8 + 1, kBf>;
            return nullptr;
    }
    return nullptr;
}

// Shapes with fused kernels: (M, C_in, C_out, bf16).  The backward keeps a
// C_in x M*C_out partial of dW per block in registers, so its list is limited
// to C_in * M * C_out <= 32768.
#define SBC_FWD_SHAPES(X) \
    X(4, 16, 32, false)   \
    X(8, 64, 64, false)   \
    X(8, 64, 128, false)  \
    X(8, 32, 32, false)   \
    X(8, 64, 64, true)    \
    X(8, 32, 32, true)
#define SBC_BWD_SHAPES(X) \
    X(4, 16, 32, false)   \
    X(8, 64, 64, false)   \
    X(8, 32, 32, false)   \
    X(8, 64, 64, true)    \
    X(8, 32, 32, true)

FwdFn find_fwd(const Shape &s, int basis_mode) {
#define SBC_X(m_, ci_, co_, bf_) \
    if (s.M == m_ && s.CI == ci_ && s.CO == co_ && s.bf == bf_) return fwd_for<m_, ci_, co_, bf_>(basis_mode);
    SBC_FWD_SHAPES(SBC_X)
#undef SBC_X
    return nullptr;
}

BwdFn find_bwd(const Shape &s, int basis_mode) {
#define SBC_X(m_, ci_, co_, bf_) \
    if (s.M == m_ && s.CI == ci_ && s.CO == co_ && s.bf == bf_) return bwd_for<m_, ci_, co_, bf_>(basis_mode);
    SBC_BWD_SHAPES(SBC_X)
#undef SBC_X
    return nullptr;
}

int basis_mode_of(const float *v, const sbc_geometry *g) {
    return v ? 0 : (int)g->basis + 1;
}

int device_cus() {
    static int cus = 0;
    if (cus == 0) {
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            cus <= 0)
            cus = 256;
    }
    return cus;
}

sbc_status launch_perm(const void *W, bool bf_in, bool bf_out, int32_t M, int32_t CI, int32_t CO,
                       int64_t s_m, int64_t s_c, int64_t s_p, void *out, hipStream_t stream) {
    const int64_t total = (int64_t)M * CI * CO;
    int64_t blocks = (total + 255) / 256;
    if (blocks > 1024) blocks = 1024;
    if (bf_out) {
        if (bf_in)
            hipLaunchKernelGGL(w_to_bf16_kernel<uint16_t>, dim3((unsigned)blocks), dim3(256), 0,
                               stream, static_cast<const uint16_t *>(W), M, CI, CO, s_m, s_c, s_p,
                               static_cast<uint16_t *>(out));
        else
            hipLaunchKernelGGL(w_to_bf16_kernel<float>, dim3((unsigned)blocks), dim3(256), 0,
                               stream, static_cast<const float *>(W), M, CI, CO, s_m, s_c, s_p,
                               static_cast<uint16_t *>(out));
    } else {
        hipLaunchKernelGGL(w_perm_f32_kernel, dim3((unsigned)blocks), dim3(256), 0, stream,
                           static_cast<const float *>(W), M, CI, CO, s_m, s_c, s_p,
                           static_cast<float *>(out));
    }
    SBC_LAUNCH_CHECK();
    return SBC_OK;
}

}  // namespace

// every listed shape has all basis variants of its M, so availability
// depends on the shape only
bool fused_forward_available(int32_t M, int32_t CI, int32_t CO, bool bf) {
    return find_fwd(Shape{M, CI, CO, bf}, 0) != nullptr;
}

bool fused_backward_available(int32_t M, int32_t CI, int32_t CO, bool bf) {
    return find_bwd(Shape{M, CI, CO, bf}, 0) != nullptr;
}

size_t fused_workspace_bytes(int32_t M, int32_t CI, int32_t CO) {
    // a permuted copy of W plus the per-block dW partials
    return align_up((size_t)M * CI * CO * 4) +
           align_up((size_t)kMaxBlocksBwd * (size_t)CI * M * CO * 4);
}

sbc_status fused_forward(const sbc_csr *csr, const float *v, const sbc_geometry *g, int32_t M,
                         const void *F, const void *W, bool bf, int32_t CI, int32_t CO, float *Y,
                         void *ws, hipStream_t stream) {
    FwdFn fn = find_fwd(Shape{M, CI, CO, bf}, basis_mode_of(v, g));
    if (!fn) return fail(SBC_ERR_UNSUPPORTED, "no fused forward for this shape");
    if (csr->n_rows == 0) return SBC_OK;
    const void *Wop = W;
    if (bf) {  // [CO, K] bf16: element (m, c, p) at p*K + m*CI + c
        const int64_t K = (int64_t)M * CI;
        SBC_TRY(launch_perm(W, true, true, M, CI, CO, CI, 1, K, ws, stream));
        Wop = ws;
    }
    const int K = M * CI;
    const int TR = (K * (bf ? 2 : 4) * 64 <= 65536) ? 64 : 32;
    sbc_geometry gg = g ? *g : sbc_geometry{};
    trace_before("fwd_fused", stream);
    hipLaunchKernelGGL(fn, dim3(grid_for(csr->n_rows, TR)), dim3(256), 0, stream, csr->n_rows,
                       csr->row_ptr, csr->col_idx, v, gg, F, Wop, Y);
    SBC_LAUNCH_CHECK();
    trace_after("fwd_fused", stream);
    return SBC_OK;
}

sbc_status fused_backward(const sbc_csr *csr, const sbc_csc *csc, const float *v,
                          const sbc_geometry *g, int32_t M, const void *F, const void *W,
                          const void *dY, bool bf, int32_t CI, int32_t CO, float *dF, float *dW,
                          void *ws, hipStream_t stream) {
    BwdFn fn = find_bwd(Shape{M, CI, CO, bf}, basis_mode_of(v, g));
    if (!fn) return fail(SBC_ERR_UNSUPPORTED, "no fused backward for this shape");
    const int32_t n_in = csr->n_cols;
    const int64_t K2 = (int64_t)M * CO;
    char *base = static_cast<char *>(ws);
    void *wt = base;
    float *part = reinterpret_cast<float *>(base + align_up((size_t)M * CI * CO * 4));
    // Wt: float32 [K2, CI] (element (m,c,p) at (m*CO + p)*CI + c), or bf16 [CI, K2]
    if (bf)
        SBC_TRY(launch_perm(W, true, true, M, CI, CO, CO, K2, 1, wt, stream));
    else
        SBC_TRY(launch_perm(W, false, false, M, CI, CO, (int64_t)CO * CI, 1, CI, wt, stream));
    const int TR = (K2 * (bf ? 2 : 4) * 64 <= 65536) ? 64 : 32;
    const int32_t n_tiles = (n_in + TR - 1) / TR;
    int blocks = device_cus();
    if (blocks > kMaxBlocksBwd) blocks = kMaxBlocksBwd;
    if (blocks > n_tiles) blocks = n_tiles;
    if (blocks < 1) blocks = 1;
    sbc_geometry gg = g ? *g : sbc_geometry{};
    if (n_in > 0 && (dF || dW)) {
        trace_before("bwd_fused", stream);
        hipLaunchKernelGGL(fn, dim3(blocks), dim3(256), 0, stream, n_in, n_tiles, csc->col_ptr,
                           csc->row_idx, csc->edge_perm, v, gg, F, dY, wt, dF,
                           dW ? part : nullptr);
        SBC_LAUNCH_CHECK();
        trace_after("bwd_fused", stream);
    }
    if (!dW) return SBC_OK;
    const int64_t total = (int64_t)M * CI * CO;
    const int64_t rb = (total + 31) / 32;
    trace_before("bwd_dw_reduce", stream);
    hipLaunchKernelGGL(dw_reduce_kernel, dim3((unsigned)rb), dim3(256), 0, stream, part,
                       n_in > 0 ? blocks : 0, M, CI, CO, dW);
    SBC_LAUNCH_CHECK();
    trace_after("bwd_dw_reduce", stream);
    return SBC_OK;
}

}  // namespace sbc
