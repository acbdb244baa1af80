// Fused kernels of the sparse basis convolution (Section 3.1: Y = sum_m
// N^(m) F W^(m), evaluated as (N F) W; its backward as the transposed
// products).  The basis values are evaluated inside the kernels from the
// coordinates (the paper computes them on the accelerator from the neighbour
// indices), or read from a materialised [E, M] array.
//
// Forward, one block per tile of TR output rows:
//   gather   G[r, m*C_in + c] = sum_e v[e, m] F[j(e), c] into LDS.  The
//            wave's edges are staged 64 at a time (index and basis values,
//            one edge per lane) in LDS; every row is owned by LPR lanes that
//            accumulate M x VEC values while walking the row's edges, loading
//            VEC contiguous channels of F[j] per edge (16-byte loads);
//   contract Y_tile = G_tile W on the matrix cores (float32: 16x16x4 f32
//            MFMA with W read from L2; bf16: G rounded to bf16 in LDS and
//            16x16x32 bf16 MFMA against a [C_out, M*C_in] copy of W).
// Forward for narrow inputs (C_in <= 32, or 64 in bf16), persistent blocks of 8 waves: each
//            wave owns 16-row tiles and keeps G in registers as the MFMA A
//            operand; W stays in LDS for the life of the block.  A row's four
//            lanes take four edges per step, with the next step's neighbour
//            indices already loaded.
// Backward (D-route), persistent blocks over tiles of 32 input rows, with
// the waves split in two roles and the tiles double-buffered in LDS:
//   gather waves   D[j, m*C_out + p] = sum_{e=(i,j)} v[e, m] dY[i, p] through
//                  the transposed pattern (and F's tile rows) for tile s+1;
//   matrix waves   dF_tile = D_tile Wt (Wt[(m, p), c] = W[m, c, p], read in
//                  place: 8 consecutive (m, p) are 8 consecutive floats of W)
//                  and dW += F_tile^T D_tile for tile s; the dW partials stay in
//                  registers and are summed afterwards in block order, so dW
//                  does not depend on scheduling.
// Sums over edges run in pattern order inside a lane; no floating-point
// atomics are used anywhere.
#include <cstdlib>
#include <type_traits>
#include <utility>

#include "basis.hpp"
#include "common.hpp"
#include "fused.hpp"
#include "spmm.hpp"

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

// Eight bf16 values p[0], p[s], ..., p[7 s] of a row-major LDS tile, as one
// MFMA operand of eight consecutive k (the k index runs down a column).
__device__ __forceinline__ bf16x8 lds_column8(const uint16_t *p, int s) {
    typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
    u16x8 r;
#pragma unroll
    for (int q = 0; q < 8; ++q) r[q] = p[q * s];
    return __builtin_bit_cast(bf16x8, r);
}

// ---------------------------------------------------------------- geometry
// Geometry as the fused kernels read it: the caller's point coordinates, and
// for event streams a packed copy (px, py, t, 0) per event, so that one
// 16-byte load brings all three coordinates of an edge's far end (three
// separate arrays would cost three cache lines per edge).
struct KGeo {
    double inv_r;
    float inv_tau;
    int32_t nnz;  // edge bound of the pattern: row extents are clamped to [0, nnz]
    const float *x_in, *x_out;
    const int4 *ev;
    const float *decays;  // learned-decay rates [8, M / 8]
};

// Basis mode of the fused kernels for the derivatives of the learned-decay
// basis with respect to its rates (the decay gradient's D-route pass).
constexpr int kDecayDerivMode = 16;

// Basis mode of the backward for the fixed-decay event basis when the
// gathered rows, the packed events or the pattern arrays pass 4 GiB: the
// generic gather (64-bit addressing) instead of the one-hot gather, whose
// loads take 32-bit byte offsets from their arrays' bases.
constexpr int kEvent8WideMode = 17;
// The same for the learned-decay basis and its derivatives (M / 8 values per
// edge), whose in-place gather takes 32-bit byte offsets too.
constexpr int kDecaysWideMode = 18;
constexpr int kDecayDerivWideMode = 19;

__global__ void pack_events_kernel(const int32_t *__restrict__ px, const int32_t *__restrict__ py,
                                   const int32_t *__restrict__ t, int32_t n,
                                   int4 *__restrict__ out) {
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
        out[i] = make_int4(px[i], py[i], t[i], 0);
}

// ---------------------------------------------------------------- basis per edge
// kBasis: 0 = read v[ev, :], SBC_BASIS_MONO4 + 1, SBC_BASIS_MONO8 + 1, SBC_BASIS_EVENT8 + 1,
// SBC_BASIS_EVENT_DECAYS + 1 (M / 8 rates per offset), kDecayDerivMode (their
// derivatives with respect to the rates) (i = output index, j = input index
// of the edge, ev = its CSR position).
template <int M, int kBasis>
__device__ __forceinline__ void edge_basis(const KGeo &g, const float *__restrict__ v,
                                           int32_t i, int32_t j, int64_t ev, double inv_r,
                                           float inv_tau, float *out) {
    if constexpr (kBasis == 0) {
#pragma unroll
        for (int m = 0; m < M; ++m) out[m] = v[ev * M + m];
    } else if constexpr (kBasis == SBC_BASIS_EVENT8 + 1 || kBasis == kEvent8WideMode) {
        const int4 a = g.ev[i], b = g.ev[j];
        const int k = event_index(a.x - b.x, a.y - b.y);
        const float d = event_decay(a.z, b.z, inv_tau);
#pragma unroll
        for (int m = 0; m < M; ++m) out[m] = (m == k) ? d : 0.f;
    } else if constexpr (kBasis == SBC_BASIS_EVENT_DECAYS + 1 || kBasis == kDecayDerivMode) {
        // the same expression as the basis values kernel, so the values agree bitwise
        constexpr int Mv = M / 8;
        const int4 a = g.ev[i], b = g.ev[j];
        const int k = event_index(a.x - b.x, a.y - b.y);
        const float dt = (float)((int64_t)a.z - (int64_t)b.z);
        float x[Mv];
#pragma unroll
        for (int q = 0; q < Mv; ++q) {
            x[q] = k >= 0 ? expf(-g.decays[k * Mv + q] * dt) : 0.f;
            if (kBasis == kDecayDerivMode) x[q] = -dt * x[q];
        }
#pragma unroll
        for (int m = 0; m < M; ++m) out[m] = (m / Mv == k) ? x[m % Mv] : 0.f;
    } else {
        point_basis<M>(g.x_out[3 * (int64_t)i], g.x_out[3 * (int64_t)i + 1],
                       g.x_out[3 * (int64_t)i + 2], g.x_in[3 * (int64_t)j],
                       g.x_in[3 * (int64_t)j + 1], g.x_in[3 * (int64_t)j + 2], inv_r, out);
    }
}

// Per-wave LDS stage of up to 64 edges: neighbour index and basis values,
// plus the row bounds of the wave's rows.
// Entry 64 is a padding edge of weight zero (its neighbour index is any valid
// row), so groups of edges can be processed without predication.
template <int M>
struct EdgeStage {
    int32_t nb[65];
    float v[65][M];
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

// The same 16 bytes kept as loaded (four registers for 8 bf16 or 4 float32
// channels), converted where they are used: twice the bf16 edges in flight
// for the registers of the converted form.
template <bool kXbf>
using RawVec = typename std::conditional<kXbf, uint4, float4>::type;

template <int C, int VEC, bool kXbf>
__device__ __forceinline__ RawVec<kXbf> load_row_raw(const void *__restrict__ Xv, int32_t r,
                                                     int cg) {
    if constexpr (kXbf)
        return *reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(Xv) +
                                                (int64_t)r * C + cg * VEC);
    else
        return *reinterpret_cast<const float4 *>(static_cast<const float *>(Xv) +
                                                 (int64_t)r * C + cg * VEC);
}

// channel k (compile-time) of a raw row vector, as float32
template <bool kXbf, int k>
__device__ __forceinline__ float raw_elem(const RawVec<kXbf> &v) {
    if constexpr (kXbf) {
        const uint32_t wd = k / 2 == 0 ? v.x : k / 2 == 1 ? v.y : k / 2 == 2 ? v.z : v.w;
        return __uint_as_float((k & 1) ? (wd & 0xFFFF0000u) : (wd << 16));
    } else {
        return k == 0 ? v.x : k == 1 ? v.y : k == 2 ? v.z : v.w;
    }
}

template <bool kXbf, int VEC, int M, int... K>
__device__ __forceinline__ void fma_row(float (&acc)[M][VEC], const RawVec<kXbf> &f, float vm,
                                        int m, std::integer_sequence<int, K...>) {
    ((acc[m][K] += vm * raw_elem<kXbf, K>(f)), ...);
}

// Row bound ptr[row_begin + lane] (clamped to [0, n_rows]) for lanes 0..RPW:
// what gather_rows needs to start, loadable one call ahead.
template <int RPW>
__device__ __forceinline__ int32_t load_bound(const int32_t *__restrict__ ptr, int32_t n_rows,
                                              int32_t row_begin, int32_t nnz) {
    const int lane = threadIdx.x & 63;
    if (lane > RPW) return 0;
    int32_t r = row_begin + lane;
    r = r < n_rows ? r : n_rows;
    r = r > 0 ? r : 0;
    const int32_t b = ptr[r];
    return b < 0 ? 0 : (b < nnz ? b : nnz);
}

// Gather of one wave's RPW consecutive rows into an LDS tile.
//   kT: the pattern is transposed (rows are inputs j, idx gives outputs i).
//   X [*, C] features gathered along the pattern; out tile row stride S
//   (elements), row r_local at out + r_local * S, column m*C + c.
//   pre.bound: load_bound<RPW>(ptr, n_rows, row_begin) of this lane;
//   pre.idx0 (pre.have_idx, pipelined only): idx[first edge + lane].
//   next_row_begin >= 0: the bound of the next call's rows (and, pipelined,
//   its first neighbour indices) is loaded while this one runs and returned.
// The wave's edges are staged 64 at a time; the rows are owned by groups of
// LPR lanes (each group owns NB rows, all accumulators live across the
// staging chunks).  kPipelined: the group's NB rows advance together with
// NB * U feature loads in flight, and the first feature loads of a chunk are
// issued together with the coordinate loads of the chunk's basis values, so
// they share one memory round trip (for persistent waves that gather while
// other waves multiply).  Otherwise the rows are taken one after another,
// four edges at a time, after the basis values (for blocks that gather and
// then multiply, where the co-resident block hides the latency).
// What a gather call hands to the next one: the next rows' bound for this
// lane and, when known, the neighbour index of the lane's edge in the next
// rows' first chunk.
struct GatherAhead {
    int32_t bound;
    int32_t idx0;
    bool have_idx;
};

template <int M, int C, int kBasis, bool kXbf, bool kOutBf, bool kT, int RPW, bool kPipelined>
__device__ __forceinline__ GatherAhead gather_rows(int32_t row_begin, int32_t n_rows,
                                                   const int32_t *__restrict__ ptr,
                                                   const int32_t *__restrict__ idx,
                                                   const int32_t *__restrict__ perm,
                                                   const float *__restrict__ v, const KGeo &g,
                                                   const void *__restrict__ Xv, void *out_tile,
                                                   int S, int local_row0, EdgeStage<M> &st,
                                                   double inv_r, float inv_tau, GatherAhead pre,
                                                   int32_t next_row_begin) {
    constexpr int VEC = kXbf ? 8 : 4;
    static_assert(C % VEC == 0, "channels must be a multiple of the vector width");
    constexpr int LPR = C / VEC;                   // lanes per row
    static_assert(LPR <= 64 && 64 % LPR == 0, "row must fit a wave");
    static_assert(RPW <= 16, "row bounds stage holds 17 entries");
    constexpr int RPB_ = 64 / LPR;
    constexpr int RPB = RPB_ < RPW ? RPB_ : RPW;   // rows in flight at once
    constexpr int NB = (RPW + RPB - 1) / RPB;      // rows per lane group
    // pipelined, with fewer rows than lane groups: SPL groups share a row,
    // group part p taking its edges rs + p, rs + p + SPL, ...; the partial
    // sums are added across the groups at the end
    constexpr int SPL = (kPipelined && RPB_ > RPW) ? RPB_ / RPW : 1;
    // edges per row loaded together: NB * U feature loads (16 bytes each, 32
    // registers in all) in flight per lane (pipelined), or 4 per row with the
    // rows taken one after another
    constexpr int UP = 8 / NB > 1 ? 8 / NB : 1;
    constexpr int U = kPipelined ? UP : 4;
    const int lane = threadIdx.x & 63;
    const int slot = lane / LPR;
    const int cg = lane % LPR;
    const int part = slot / RPB;                   // < SPL
    const int rslot = slot % RPB;

    if (lane <= RPW) st.bounds[lane] = pre.bound;
    const int32_t next_bound =
        next_row_begin >= 0 ? load_bound<RPW>(ptr, n_rows, next_row_begin, g.nnz) : 0;
    wave_lds_sync();
    const int32_t wb = st.bounds[0], we = st.bounds[RPW];
    int32_t rs[NB], re[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        const int lr = b * RPB + rslot;
        const bool own = slot < RPB * SPL && lr < RPW;
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
        int32_t row = 0, other = 0;
        int64_t ev = 0;
        if (e < we) {
            int s = 0;
#pragma unroll
            for (int q = 1; q < RPW; ++q)
                if (st.bounds[q] <= e) s = q;
            row = row_begin + s;
            other = (kPipelined && pre.have_idx && c0 == wb) ? pre.idx0 : idx[e];
            ev = (kBasis == 0) ? (perm ? (int64_t)perm[e] : (int64_t)e) : 0;
            st.nb[lane] = other;
            if (lane == 0) st.nb[64] = other;  // padding edge: a valid row, weight 0
        }
        if constexpr (!kPipelined) {
            // basis values first, then each row of the lane group in turn
            if (e < we) {
                float bv[M];
                if (kT)
                    edge_basis<M, kBasis>(g, v, other, row, ev, inv_r, inv_tau, bv);
                else
                    edge_basis<M, kBasis>(g, v, row, other, ev, inv_r, inv_tau, bv);
#pragma unroll
                for (int m = 0; m < M; ++m) st.v[lane][m] = bv[m];
                if (lane == 0) {
#pragma unroll
                    for (int m = 0; m < M; ++m) st.v[64][m] = 0.f;
                }
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
#pragma unroll
                    for (int u = 0; u < U; ++u) {
                        q[u] = e2 + u < hi ? e2 + u - c0 : 64;
                        load_row_vec<C, VEC, kXbf>(Xv, st.nb[q[u]], cg, f[u]);
                    }
#pragma unroll
                    for (int u = 0; u < U; ++u)
#pragma unroll
                        for (int m = 0; m < M; ++m) {
                            const float vm = st.v[q[u]][m];
#pragma unroll
                            for (int k = 0; k < VEC; ++k) acc[b][m][k] += vm * f[u][k];
                        }
                }
            }
            wave_lds_sync();
            continue;
        }
        wave_lds_sync();
        // the lane group's NB rows advance together, U edges each per step
        int32_t pos[NB], hi[NB];
        int32_t steps = 0;
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            // this part's first edge at or after the chunk start
            const int32_t lo = rs[b] > c0 ? rs[b] : c0;
            const int32_t d = lo - (rs[b] + part);
            pos[b] = rs[b] + part + (d > 0 ? (d + SPL - 1) / SPL : 0) * SPL;
            hi[b] = re[b] < c0 + 64 ? re[b] : c0 + 64;
            const int32_t mine = hi[b] > pos[b] ? (hi[b] - pos[b] + SPL - 1) / SPL : 0;
            const int32_t n = (mine + U - 1) / U;
            steps = n > steps ? n : steps;
        }
        RawVec<kXbf> f[NB][U];
        int q[NB][U];
        auto issue = [&]() {
#pragma unroll
            for (int b = 0; b < NB; ++b)
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    q[b][u] = pos[b] + u * SPL < hi[b] ? pos[b] + u * SPL - c0 : 64;
                    f[b][u] = load_row_raw<C, VEC, kXbf>(Xv, st.nb[q[b][u]], cg);
                }
        };
        if (steps > 0) issue();
        // basis values of this lane's edge; their coordinate loads overlap the
        // feature loads just issued
        if (e < we) {
            float bv[M];
            if (kT)
                edge_basis<M, kBasis>(g, v, other, row, ev, inv_r, inv_tau, bv);
            else
                edge_basis<M, kBasis>(g, v, row, other, ev, inv_r, inv_tau, bv);
#pragma unroll
            for (int m = 0; m < M; ++m) st.v[lane][m] = bv[m];
            if (lane == 0) {
#pragma unroll
                for (int m = 0; m < M; ++m) st.v[64][m] = 0.f;
            }
        }
        wave_lds_sync();
#pragma unroll 1
        for (int32_t it = 0; it < steps; ++it) {
            if (it > 0) issue();
#pragma unroll
            for (int b = 0; b < NB; ++b) {
#pragma unroll
                for (int u = 0; u < U; ++u)
#pragma unroll
                    for (int m = 0; m < M; ++m)
                        fma_row<kXbf, VEC>(acc[b], f[b][u], st.v[q[b][u]][m], m,
                                           std::make_integer_sequence<int, VEC>{});
                pos[b] += U * SPL;
            }
        }
        wave_lds_sync();
    }
    if constexpr (SPL > 1) {
        // add the parts of each row (every lane of the row ends with the same sum)
#pragma unroll
        for (int d = RPB * LPR; d < RPB * LPR * SPL; d <<= 1)
#pragma unroll
            for (int m = 0; m < M; ++m)
#pragma unroll
                for (int k = 0; k < VEC; ++k) acc[0][m][k] += __shfl_xor(acc[0][m][k], d, 64);
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        const int lr = b * RPB + slot;
        if (slot < RPB && lr < RPW) {
#pragma unroll
            for (int m = 0; m < M; ++m) {
                if constexpr (kOutBf) {
                    static_assert(VEC == 8, "bf16 rows are written 16 bytes at a time");
                    typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
                    u16x8 packed;
#pragma unroll
                    for (int k = 0; k < VEC; ++k) packed[k] = f2bf(acc[b][m][k]);
                    *reinterpret_cast<u16x8 *>(static_cast<uint16_t *>(out_tile) +
                                               (int64_t)(local_row0 + lr) * S + m * C +
                                               cg * VEC) = packed;
                } else {
                    float *o = static_cast<float *>(out_tile) + (int64_t)(local_row0 + lr) * S +
                               m * C + cg * VEC;
#pragma unroll
                    for (int k = 0; k < VEC; ++k) o[k] = acc[b][m][k];
                }
            }
        }
    }
    GatherAhead ahead{next_bound, 0, false};
    if (kPipelined && next_row_begin >= 0) {
        const int32_t nb0 = __shfl(next_bound, 0, 64), nb1 = __shfl(next_bound, RPW, 64);
        ahead.idx0 = nb0 + lane < nb1 ? idx[nb0 + lane] : 0;
        ahead.have_idx = true;
    }
    return ahead;
}

// ---------------------------------------------------------------- one-hot event gather
// The fixed-decay event basis (SBC_BASIS_EVENT8) has one nonzero value per
// edge, at the offset index k of its pixel step (none for a same-pixel edge),
// so a gathered row's sum over its edges only adds each edge into one of the
// M = 8 column blocks.  gather_rows_onehot builds the same tile rows as
// gather_rows without the other seven products.  A wave takes its rows'
// edges in chunks of CK (32 or 64); per chunk:
//   1. the chunk's CK neighbour rows, loaded into registers while the
//      previous chunk was summed, are written to LDS, and each edge's offset
//      index and decay come from its endpoints' coordinates (loaded with the
//      rows);
//   2. the loads of the following chunk are issued (the wave's next chunk of
//      these rows, else the first chunk of its rows in the next tile);
//   3. wave ballots of the bits of each edge's offset and row mark, for lane
//      (row r, offset m, channel part h), the chunk's edges of row r with
//      offset m (its bucket);
//   4. each lane walks the set bits of its bucket, lowest first, and adds up
//      those rows, CH channels of each, from LDS.
// So a (row, offset) sum takes its edges in pattern order, one product each,
// and a chunk's memory round trip overlaps the previous chunk's sums.  The
// indices that step 2 needs are loaded a chunk (or a tile) earlier, and the
// row bounds two tiles earlier, so no step waits on a load issued in the
// same step.
// 16 bytes as a native vector (its copies stay in registers, which those of
// the HIP uint4 struct do not always)
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int RB, int CK>  // bytes per gathered row, edges per chunk
struct OneHotStage {
    u32x4 f[CK + 1][RB / 16];   // the chunk's neighbour rows, then a row of zeros
    float sv[CK + 1];           // basis value of each staged edge, then 0
};

// The stage's row of zeros and its basis value 0, which the bucket walk
// reads past a bucket's end (so its reads need no branch).
template <int RB, int CK>
__device__ __forceinline__ void onehot_stage_init(OneHotStage<RB, CK> &st) {
    const int lane = threadIdx.x & 63;
    if (lane < RB / 16) st.f[CK][lane] = u32x4{0u, 0u, 0u, 0u};
    if (lane == 0) st.sv[CK] = 0.f;
}

// Bits [0, n) of a 64-bit lane mask.
__device__ __forceinline__ uint64_t lanes_below(int n) {
    return n >= 64 ? ~0ull : (n <= 0 ? 0ull : ((1ull << n) - 1ull));
}

// Element k of a 16-byte piece of float32 (4) or bf16 (8) values, as float32.
template <bool kBf>
__device__ __forceinline__ float piece_elem(const u32x4 &x, int k) {
    const uint32_t w = x[kBf ? k / 2 : k];
    if constexpr (kBf) return __uint_as_float((k & 1) ? (w & 0xFFFF0000u) : (w << 16));
    else return __uint_as_float(w);
}

// The one-hot gather's loads in flight from one tile to the next (per lane).
// Tile t of the wave's sequence: b0 = its row bounds (lanes 0..RPW), b1
// those of the next tile, b2 those of the one after as loaded (unclamped,
// onehot_bound_raw); j1 = idx of the next tile's first chunk (lane e: its
// edge e); i1 = idx of this tile's second chunk; rows, ga, gb = the
// neighbour-row pieces and endpoint coordinates of this tile's first chunk
// (or, inside a call, of the chunk after the one being summed).
template <int NR>  // 16-byte row pieces per lane and chunk (CK = NR RPL)
struct OneHotPipe {
    int32_t b0, b1, b2, j1, i1;
    u32x4 rows[NR];
    int4 ga, gb;
    int32_t es;  // the row (0 .. RPW-1) of the lane's edge in the chunk
};

// Row begins of the wave's tiles t .. t+3 (-1 past its last tile).
struct OneHotTiles {
    int32_t r0, r1, r2, r3;
};

// load_bound without its clamp and without a branch: every lane loads
// (lanes past RPW repeat lane RPW's row; a missing tile, row_begin < 0, reads
// from row 0), so no wait for the load lands before the value's use, where
// onehot_bound_clamp finishes it.
template <int RPW>
__device__ __forceinline__ int32_t onehot_bound_raw(const int32_t *__restrict__ ptr,
                                                    int32_t n_rows, int32_t row_begin) {
    const int lane = threadIdx.x & 63;
    int32_t r = (row_begin > 0 ? row_begin : 0) + (lane < RPW ? lane : RPW);
    r = r < n_rows ? r : n_rows;
    return ptr[r];
}

__device__ __forceinline__ int32_t onehot_bound_clamp(int32_t b, int32_t nnz) {
    return b < 0 ? 0 : (b < nnz ? b : nnz);
}

// idx of the chunk at edge c0 (lane e: edge c0 + e), loaded by every lane
// without a branch: the edge is clamped into [0, nnz) (nnz > 0), and what a
// lane past its rows' end holds is not used (onehot_issue).  (The one-hot
// gather's loads use 32-bit byte offsets: nnz * 4 < 2^32.)
__device__ __forceinline__ int32_t onehot_chunk_idx(const int32_t *__restrict__ idx, int32_t c0,
                                                    int32_t nnz) {
    int32_t e = c0 + (int32_t)(threadIdx.x & 63);
    e = e < nnz ? e : nnz - 1;
    e = e > 0 ? e : 0;
    return *reinterpret_cast<const int32_t *>(reinterpret_cast<const char *>(idx) +
                                              ((uint32_t)e << 2));
}

// Issue the loads of the chunk at edge c0 (c0 < the rows' end) of the rows
// [row_begin, row_begin + RPW) with bounds bnd and chunk indices other (from
// onehot_chunk_idx): lane l's endpoint coordinates for edge c0 + l, and row
// piece q of lane l, piece l % P of staged row q RPL + l / P.  Lanes past the
// rows' end or the chunk's CK edges load lane 0's edge, so every lane's
// addresses are in bounds.  Byte offsets from X and from the packed events
// are 32-bit (the host checks that both arrays are under 4 GiB).
template <int C, int RPW, bool kT, bool kBf, int NR>
__device__ __forceinline__ void onehot_issue(int32_t row_begin, int32_t bnd, int32_t c0,
                                             int32_t other, const KGeo &g,
                                             const void *__restrict__ X, OneHotPipe<NR> &p) {
    constexpr int ES = kBf ? 2 : 4;
    constexpr int P = C * ES / 16;     // 16-byte pieces per row
    constexpr int RPL = 64 / P;        // rows per load instruction
    constexpr int CK = NR * RPL;       // edges per chunk
    static_assert(CK == 32 || CK == 64, "chunk size");
    const int lane = threadIdx.x & 63;
    const int32_t e = c0 + lane;
    // the row of the lane's edge: the row starts (bounds 1 .. RPW-1, read as
    // wave-uniform values) at or below it
    int s = 0;
#pragma unroll
    for (int q = 1; q < RPW; ++q) s += __builtin_amdgcn_readlane(bnd, q) <= e ? 1 : 0;
    const bool has = lane < CK && e < __builtin_amdgcn_readlane(bnd, RPW);
    const int32_t other0 = __builtin_amdgcn_readlane(other, 0);
    const int32_t s0 = __builtin_amdgcn_readlane(s, 0);
    other = has ? other : other0;
    s = has ? s : s0;
    const char *Xb = static_cast<const char *>(X);
#pragma unroll
    for (int q = 0; q < NR; ++q) {
        const int32_t src = __shfl(other, q * RPL + lane / P, 64);
        p.rows[q] = *reinterpret_cast<const u32x4 *>(
            Xb + ((uint32_t)src * (uint32_t)(C * ES) + (uint32_t)(16 * (lane % P))));
    }
    const int32_t row = row_begin + s;
    const char *evb = reinterpret_cast<const char *>(g.ev);
    p.ga = *reinterpret_cast<const int4 *>(evb + ((uint32_t)(kT ? other : row) << 4));
    p.gb = *reinterpret_cast<const int4 *>(evb + ((uint32_t)(kT ? row : other) << 4));
    p.es = s;
}

// The pipeline's start for the wave's first tile (rows at tl.r0 >= 0).
template <int C, int RPW, bool kT, bool kBf, int NR>
__device__ __forceinline__ void onehot_prologue(const OneHotTiles &tl, int32_t n_rows,
                                                const int32_t *__restrict__ ptr,
                                                const int32_t *__restrict__ idx, const KGeo &g,
                                                const void *__restrict__ X, OneHotPipe<NR> &p) {
    p.b0 = load_bound<RPW>(ptr, n_rows, tl.r0, g.nnz);
    p.b1 = tl.r1 >= 0 ? load_bound<RPW>(ptr, n_rows, tl.r1, g.nnz) : 0;
    p.b2 = onehot_bound_raw<RPW>(ptr, n_rows, tl.r2);
    p.i1 = p.j1 = 0;
    if (g.nnz == 0) return;  // no edges in any tile
    const int32_t wb = __shfl(p.b0, 0, 64), we = __shfl(p.b0, RPW, 64);
    constexpr int CK = NR * (64 / (C * (kBf ? 2 : 4) / 16));
    const int32_t i0 = onehot_chunk_idx(idx, wb, g.nnz);
    p.i1 = onehot_chunk_idx(idx, wb + CK, g.nnz);
    p.j1 = onehot_chunk_idx(idx, __shfl(p.b1, 0, 64), g.nnz);
    if (wb < we) onehot_issue<C, RPW, kT, kBf, NR>(tl.r0, p.b0, wb, i0, g, X, p);
}

// X [*, C] float32 or bf16 (kBf), tile rows of the same type.  p holds the
// state described at OneHotPipe for tile tl.r0 and is advanced to the next.
template <int C, int RPW, bool kT, bool kBf, int NR>
__device__ __forceinline__ void gather_rows_onehot(
    const OneHotTiles &tl, int32_t n_rows, const int32_t *__restrict__ ptr,
    const int32_t *__restrict__ idx, const KGeo &g, const void *__restrict__ X, void *out_tile,
    int S, int local_row0, OneHotStage<C * (kBf ? 2 : 4), NR * (64 / (C * (kBf ? 2 : 4) / 16))> &st,
    float inv_tau, OneHotPipe<NR> &p) {
    constexpr int M = 8;
    constexpr int ES = kBf ? 2 : 4;            // bytes per element
    constexpr int VPP = 16 / ES;               // values per 16-byte piece
    constexpr int H = 64 / (RPW * M);          // lanes sharing a bucket (channel parts)
    static_assert(H >= 1 && RPW * M * H == 64 && RPW <= 16, "a lane per (row, offset, part)");
    constexpr int CH = C / H;                  // channels per lane
    static_assert(CH % VPP == 0, "whole 16-byte pieces per lane");
    constexpr int NP = CH / VPP;               // 16-byte pieces per lane
    constexpr int P = C / VPP;                 // 16-byte pieces per row
    static_assert(64 % P == 0, "whole rows per load instruction");
    constexpr int RPL = 64 / P;                // rows per load instruction
    constexpr int CK = NR * RPL;               // edges per chunk
    // bucket rows read together (four, with the next chunk's rows in flight in
    // registers, took more instructions per product and ran slower)
    constexpr int U = CK == 32 && NP <= 4 ? 4 : 2;
    constexpr int NPX = U * NP > 8 ? 8 / U : NP;  // pieces per row and read pass
    static_assert(NP % NPX == 0, "whole read passes");
    const int lane = threadIdx.x & 63;
    // this lane's bucket
    const int br = lane / (M * H), bm = (lane / H) % M, bh = lane % H;

    // loads for later tiles: bounds three tiles ahead, the first chunk's
    // indices two tiles ahead, the second chunk's one tile ahead.  They are
    // issued after the first chunk's rows are taken and after the next
    // chunk's loads: loads complete in issue order, so no wait for a chunk's
    // rows waits for a load issued after them
    const int32_t b2 = onehot_bound_clamp(p.b2, g.nnz);
    int32_t b3 = 0, j2 = 0, i1n = 0;
    auto ahead_loads = [&]() {
        b3 = onehot_bound_raw<RPW>(ptr, n_rows, tl.r3);
        j2 = onehot_chunk_idx(idx, __builtin_amdgcn_readlane(b2, 0), g.nnz);
        i1n = onehot_chunk_idx(idx, __builtin_amdgcn_readlane(p.b1, 0) + CK, g.nnz);
    };

    const int32_t wb = __builtin_amdgcn_readlane(p.b0, 0);
    const int32_t we = __builtin_amdgcn_readlane(p.b0, RPW);
    const int32_t nb0 = __builtin_amdgcn_readlane(p.b1, 0);
    const int32_t nb1 = __builtin_amdgcn_readlane(p.b1, RPW);
    constexpr int SB = RPW <= 1 ? 0 : RPW <= 2 ? 1 : RPW <= 4 ? 2 : RPW <= 8 ? 3 : 4;  // row bits
    float acc[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c) acc[c] = 0.f;

#pragma unroll 1
    for (int32_t c0 = wb; c0 < we; c0 += CK) {
        // 1. the chunk's rows into LDS; its edges' offsets and decays
#pragma unroll
        for (int q = 0; q < NR; ++q) st.f[q * RPL + lane / P][lane % P] = p.rows[q];
        const bool has = lane < CK && c0 + lane < we;
        const int k = has ? event_index(p.ga.x - p.gb.x, p.ga.y - p.gb.y) : -1;
        const float sv = has ? event_decay(p.ga.z, p.gb.z, inv_tau) : 0.f;
        if (lane < CK) st.sv[lane] = sv;
        const int es = p.es;
        // 2. the next chunk's loads, then (first chunk) those for later tiles
        if (c0 + CK < we) {
            onehot_issue<C, RPW, kT, kBf, NR>(tl.r0, p.b0, c0 + CK, p.i1, g, X, p);
            p.i1 = onehot_chunk_idx(idx, c0 + 2 * CK, g.nnz);
        } else if (tl.r1 >= 0 && nb0 < nb1) {
            onehot_issue<C, RPW, kT, kBf, NR>(tl.r1, p.b1, nb0, p.j1, g, X, p);
        }
        if (c0 == wb) ahead_loads();
        // 3. this lane's bucket: the chunk's edges whose offset bits equal bm's
        // and whose row bits equal br's
        uint64_t bsel = __ballot(k >= 0);
#pragma unroll
        for (int b = 0; b < 3; ++b) {
            const uint64_t v = __ballot((k >> b) & 1);
            bsel &= (bm >> b) & 1 ? v : ~v;
        }
#pragma unroll
        for (int b = 0; b < SB; ++b) {
            const uint64_t v = __ballot((es >> b) & 1);
            bsel &= (br >> b) & 1 ? v : ~v;
        }
        wave_lds_sync();
        // 4. the bucket's rows, U at a time, lowest lane first: the reads of a
        // group are issued before its products; past the bucket's end a lane
        // reads the row of zeros with weight 0
        if (__ballot(bsel != 0ull) != 0ull) do {
            int32_t li[U];  // staged edge, or CK (the row of zeros) past the bucket's end
#pragma unroll
            for (int u = 0; u < U; ++u) {
                li[u] = bsel != 0ull ? (int32_t)__builtin_ctzll(bsel) : CK;
                bsel &= bsel - 1ull;
            }
            float vv[U];
#pragma unroll
            for (int u = 0; u < U; ++u) vv[u] = st.sv[li[u]];
            // the pieces in passes of NPX (eight 16-byte reads in flight), in an
            // order rotated by the offset, so the lanes of one LDS cycle read
            // different banks (rows are 128 B apart)
#pragma unroll
            for (int c0p = 0; c0p < NP; c0p += NPX) {
                u32x4 x[U][NPX];
#pragma unroll
                for (int u = 0; u < U; ++u)
#pragma unroll
                    for (int c = 0; c < NPX; ++c)
                        x[u][c] = st.f[li[u]][bh * NP + (c0p + c + bm) % NP];
#pragma unroll
                for (int u = 0; u < U; ++u)
#pragma unroll
                    for (int c = 0; c < NPX; ++c)
#pragma unroll
                        for (int q = 0; q < VPP; ++q)
                            acc[VPP * (c0p + c) + q] += vv[u] * piece_elem<kBf>(x[u][c], q);
            }
        } while (__ballot(bsel != 0ull) != 0ull);
        wave_lds_sync();  // the stage is rewritten by the next chunk
    }
    // rows without edges: the next tile's first chunk, and the loads ahead
    if (wb >= we) {
        if (tl.r1 >= 0 && nb0 < nb1)
            onehot_issue<C, RPW, kT, kBf, NR>(tl.r1, p.b1, nb0, p.j1, g, X, p);
        if (g.nnz > 0) ahead_loads();
    }
    // this lane's (row, offset, part) block of the tile row; piece c of acc is
    // piece (c + bm) % NP of the block
    char *o = static_cast<char *>(out_tile) +
              ((int64_t)(local_row0 + br) * S + bm * C + bh * CH) * ES;
#pragma unroll
    for (int c = 0; c < NP; ++c) {
        u32x4 v;
#pragma unroll
        for (int q = 0; q < 4; ++q)
            v[q] = kBf ? (uint32_t)f2bf(acc[VPP * c + 2 * q]) |
                             ((uint32_t)f2bf(acc[VPP * c + 2 * q + 1]) << 16)
                       : __float_as_uint(acc[VPP * c + q]);
        *reinterpret_cast<u32x4 *>(o + 16 * ((c + bm) % NP)) = v;
    }
    p.b0 = p.b1;
    p.b1 = b2;
    p.b2 = b3;
    p.j1 = j2;
    p.i1 = i1n;
}

// f(std::integral_constant<int, s>) for s = 0 .. N - 1, unrolled whatever
// the body's size (register arrays indexed by s stay in registers)
template <typename F, int... S>
__device__ __forceinline__ void static_for_impl(F &&f, std::integer_sequence<int, S...>) {
    (f(std::integral_constant<int, S>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F &&f) {
    static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// One-hot gather of the transposed pattern into the D tile in place, for
// rows of 32 float32 channels and RPW = 4 or 8 rows per wave: the LPR = 64 /
// RPW lanes of a row each own CO / LPR channels of it for all offsets and add
// every edge of the row into those channels at the edge's offset (an LDS
// read, the FMAs and a write; no stage, no ballots and no bucket walk, which
// frees the LDS for tiles of 64 rows).  The lanes of a row load one neighbour
// row, 128 contiguous bytes, per step.  Edges come in chunks of LPR per row
// (at least one chunk per tile): lane p takes index, coordinates, offset and
// decay of edge p of the chunk, broadcast to the row's lanes by DPP.  Rows of
// a wave have their own lanes, so no two lanes write one address; LDS
// accesses of one wave complete in order, so consecutive edges of one offset
// chain correctly.
//
// The chunks of the wave's tiles form one stream, across the block barrier:
// a chunk's neighbour rows are loaded during the chunk before it (step s of
// chunk c loads the row of step s of chunk c + 1 into the register it has
// just used), its coordinates at the start of the chunk before, and its
// indices two chunks ahead; row bounds come three tiles ahead.
template <int LPR>
struct RmwPipe {
    int32_t e0a, e1a, e0b, e1b, e0c, e1c;  // bounds of this lane's row in tiles s, s + 1, s + 2
    int32_t C0, C1, S0;    // chunks of tiles s and s + 1, steps of tile s (wave-uniform)
    int4 bc, bn;           // coordinates of the row in tiles s and s + 1
    int32_t i1;            // index of edge p of the next chunk (in flight until used)
    bool v1;               // whether that edge lies inside its row
    int4 ev1;              // coordinates of the next chunk's neighbours (in flight)
    using PT = typename std::conditional<LPR == 16, float2, float4>::type;
    PT y[LPR];             // the lane's pieces of the current chunk's rows (in flight)
};

// The edge's basis: kValues 0, the fixed decay exp(-dt / tau) (one value per
// edge); 1, the learned decays exp(-lambda_{k,q} dt) (MV values per edge, at
// slots k MV + q); 2, their derivatives -dt exp(-lambda_{k,q} dt).
template <int CO, int RPW, int MV = 1, int kValues = 0>
struct RmwGather {
    static constexpr int LPR = 64 / RPW;  // lanes per row
    static constexpr int CH = CO / LPR;   // channels per lane
    static_assert(CO == 32 && (RPW == 4 || RPW == 8), "rows of 32 float32 channels");
    static_assert(kValues == 0 ? MV == 1 : MV >= 1, "values per edge");
    static constexpr int kMV = MV, kVal = kValues;
    using PT = typename RmwPipe<LPR>::PT;
    using Pipe = RmwPipe<LPR>;
    const int32_t *ptr, *idx;
    const int4 *ev;
    const float *X;
    const float *decays;  // [8, MV] (kValues 1 and 2)
    int32_t n_rows, nnz;
    float inv_tau;
    int r, p;

    __device__ __forceinline__ void bounds_raw(int32_t row_begin, int32_t &b0, int32_t &b1) const {
        const int32_t row = row_begin + r;
        const int32_t q = row_begin >= 0 && row < n_rows ? row : 0;
        b0 = ptr[q];
        b1 = ptr[q + 1];
    }
    __device__ __forceinline__ void clamp(int32_t row_begin, int32_t b0, int32_t b1, int32_t &e0,
                                          int32_t &e1) const {
        const bool ok = row_begin >= 0 && row_begin + r < n_rows;
        b0 = b0 < 0 ? 0 : (b0 < nnz ? b0 : nnz);
        b1 = b1 < b0 ? b0 : (b1 < nnz ? b1 : nnz);
        e0 = ok ? b0 : 0;
        e1 = ok ? b1 : 0;
    }
    // steps (the longest row's edges) of a tile, and its chunks (at least 1)
    __device__ __forceinline__ int32_t steps(int32_t e0, int32_t e1) const {
        int32_t len = e1 - e0;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int32_t o = __shfl_xor(len, d, 64);
            len = o > len ? o : len;
        }
        return __builtin_amdgcn_readfirstlane(len);
    }
    static __device__ __forceinline__ int32_t chunks(int32_t S) {
        return S > LPR ? (S + LPR - 1) / LPR : 1;
    }
    __device__ __forceinline__ int4 coords(int32_t row_begin) const {
        const int32_t row = row_begin + r;
        return ev[row_begin >= 0 && row < n_rows ? row : 0];
    }
    // (nnz >= 1: the host takes this gather only then; positions are clamped
    // into [0, nnz) and the value is used only inside the row)
    __device__ __forceinline__ int32_t idx_raw(int32_t e) const {
        return idx[e < nnz ? e : nnz - 1];
    }
    // value v of lane s of this lane's row (a DPP broadcast within the 16
    // lanes of a DPP row: a plain VALU move, where a cross-lane read through
    // LDS took a round trip; with 8 lanes per row, the upper 8 of a DPP row
    // take lane 8 + s)
    template <int S>
    static __device__ __forceinline__ int32_t row_lane(int32_t v) {
        if constexpr (LPR == 16) {
            return __builtin_amdgcn_mov_dpp(v, 0x150 + S, 0xf, 0xf, false);
        } else {
            const int32_t lo = __builtin_amdgcn_mov_dpp(v, 0x150 + S, 0xf, 0xf, false);
            const int32_t hi = __builtin_amdgcn_mov_dpp(v, 0x158 + S, 0xf, 0xf, false);
            return (threadIdx.x & 8) ? hi : lo;
        }
    }
    // (32-bit byte offsets: the host takes this gather while the gathered
    // rows are under 4 GiB)
    template <int S>
    __device__ __forceinline__ void load_row(int32_t i, PT &yv) const {
        const uint32_t j = (uint32_t)row_lane<S>(i);
        yv = *reinterpret_cast<const PT *>(reinterpret_cast<const char *>(X) +
                                           (j * (uint32_t)(CO * 4) + 4 * CH * p));
    }
    // the indices of the chunk two ahead of chunk c of tile s
    __device__ __forceinline__ void issue_idx(Pipe &P, int32_t c) const {
        int32_t t = c + 2, tt = 0;
        if (t >= P.C0) {
            t -= P.C0;
            tt = 1;
            if (t >= P.C1) {
                t -= P.C1;
                tt = 2;
            }
        }
        // (as differences: a select between two members became a load through
        // a selected address, which kept the whole pipe in memory)
        const int32_t e0 = P.e0a + (tt >= 1 ? P.e0b - P.e0a : 0) + (tt >= 2 ? P.e0c - P.e0b : 0);
        const int32_t e1 = P.e1a + (tt >= 1 ? P.e1b - P.e1a : 0) + (tt >= 2 ? P.e1c - P.e1b : 0);
        const int32_t e = e0 + LPR * t + p;
        P.i1 = idx_raw(e);
        P.v1 = e < e1;
    }
};

// Before the first tile (rows rb0 .. rb2 of tiles 0 .. 2): their bounds, the
// loads of the first chunk and the indices of the second.
template <class G_>
__device__ __forceinline__ void rmw_prologue(const G_ &G, int32_t rb0, int32_t rb1, int32_t rb2,
                                             typename G_::Pipe &P) {
    int32_t b0, b1;
    G.bounds_raw(rb0, b0, b1);
    G.clamp(rb0, b0, b1, P.e0a, P.e1a);
    G.bounds_raw(rb1, b0, b1);
    G.clamp(rb1, b0, b1, P.e0b, P.e1b);
    G.bounds_raw(rb2, b0, b1);
    G.clamp(rb2, b0, b1, P.e0c, P.e1c);
    P.S0 = G.steps(P.e0a, P.e1a);
    P.C0 = G.chunks(P.S0);
    P.C1 = G.chunks(G.steps(P.e0b, P.e1b));
    P.bc = G.coords(rb0);
    P.bn = G.coords(rb1);
    const int32_t e = P.e0a + G.p;
    int32_t i0 = G.idx_raw(e);
    i0 = e < P.e1a ? i0 : 0;
    {  // the second chunk: chunk 1 of tile 0, or chunk 0 of tile 1
        const bool nt = P.C0 < 2;
        const int32_t e0 = P.e0a + (nt ? P.e0b - P.e0a : G_::LPR),
                      e1 = P.e1a + (nt ? P.e1b - P.e1a : 0);
        P.i1 = G.idx_raw(e0 + G.p);
        P.v1 = e0 + G.p < e1;
    }
    P.ev1 = G.ev[i0];
    static_for<G_::LPR>(
        [&](auto sc) { G.template load_row<decltype(sc)::value>(i0, P.y[sc.value]); });
}

// Tile s of the stream into the wave's rows of out_tile (row_begin: the
// wave's first row in tile s; rb2, rb3: in tiles s + 2, s + 3; -1 where there
// is none).
template <class G_>
__device__ __forceinline__ void gather_rows_rmw(const G_ &G, int32_t rb2, int32_t rb3,
                                                float *out_tile, int SD, int local_row0,
                                                typename G_::Pipe &P) {
    constexpr int LPR = G_::LPR, CH = G_::CH, CO = G_::CH * G_::LPR, MV = G_::kMV;
    using PT = typename G_::PT;
    const int r = G.r, p = G.p;
    float *drow = out_tile + (local_row0 + r) * SD;
    // (the row's 8 MV CO values, 4 LPR floats per 16-byte store of its lanes)
#pragma unroll
    for (int q = 0; q < 8 * MV * CO / (4 * LPR); ++q)
        *reinterpret_cast<float4 *>(drow + 4 * LPR * q + 4 * p) = make_float4(0.f, 0.f, 0.f, 0.f);
    // the tile pipeline: bounds of tile s + 3, coordinates of the rows of s + 2
    int32_t b0n, b1n;
    G.bounds_raw(rb3, b0n, b1n);
    const int4 bnn = G.coords(rb2);
    const int4 bc = P.bc;
#pragma unroll 1
    for (int32_t c = 0; c < P.C0; ++c) {
        // this chunk: offset and basis values of edge p of the row (its
        // coordinates were loaded at the start of the chunk before), in the
        // expressions of the basis values kernel, so the values agree bitwise
        const int4 a = P.ev1;
        const int k = event_index(a.x - bc.x, a.y - bc.y);
        float d[MV];
        if constexpr (G_::kVal == 0) {
            d[0] = event_decay(a.z, bc.z, G.inv_tau);
        } else {
            const float dt = (float)((int64_t)a.z - (int64_t)bc.z);
            const int kk = k >= 0 ? k : 0;
#pragma unroll
            for (int q = 0; q < MV; ++q) {
                d[q] = expf(-G.decays[kk * MV + q] * dt);
                if constexpr (G_::kVal == 2) d[q] = -dt * d[q];
            }
        }
        const int32_t e = P.e0a + LPR * c + p;
        const bool live = e < P.e1a && k >= 0;
        const int32_t koff = live ? k * MV * CO : 0;
#pragma unroll
        for (int q = 0; q < MV; ++q) d[q] = live ? d[q] : 0.f;
        // the next chunk: its indices (loaded a chunk ago), its coordinates
        // now and its rows step by step below; the indices of the one after
        const int32_t i1 = P.v1 ? P.i1 : 0;
        P.ev1 = G.ev[i1];
        G.issue_idx(P, c);
        const int32_t ns = P.S0 - LPR * c;
        static_for<LPR>([&](auto sc) {
            constexpr int s = decltype(sc)::value;
            if (s < ns) {
                const int32_t o = G_::template row_lane<s>(koff);
#pragma unroll
                for (int v = 0; v < MV; ++v) {
                    const float dd =
                        __int_as_float(G_::template row_lane<s>(__float_as_int(d[v])));
                    PT *q = reinterpret_cast<PT *>(drow + o + v * CO + CH * p);
                    PT acc = *q;
                    acc.x = fmaf(dd, P.y[s].x, acc.x);
                    acc.y = fmaf(dd, P.y[s].y, acc.y);
                    if constexpr (CH == 4) {
                        acc.z = fmaf(dd, P.y[s].z, acc.z);
                        acc.w = fmaf(dd, P.y[s].w, acc.w);
                    }
                    *q = acc;
                }
            }
            G.template load_row<s>(i1, P.y[s]);
        });
    }
    // the next tile
    P.e0a = P.e0b;
    P.e1a = P.e1b;
    P.e0b = P.e0c;
    P.e1b = P.e1c;
    G.clamp(rb3, b0n, b1n, P.e0c, P.e1c);
    P.C0 = P.C1;
    P.S0 = G.steps(P.e0a, P.e1a);
    P.C1 = G.chunks(G.steps(P.e0b, P.e1b));
    P.bc = P.bn;
    P.bn = bnn;
}

// acc[u][t] += A_tile[16 rb_u .., :] x B[:, 16 cb_t ..] for the 16x16 blocks of
// one wave (rb_u = wr + NRG u, cb_t = wc + NCBW t).  A sits in LDS (row stride
// S elements), B in global memory as B^T [NCOL, K].  The B fragments of
// k-groups alternate between two register sets, so the loads of the next
// group are in flight while the current group is multiplied (no copies
// between the sets, which would force a wait).
//
// float32 variant with B given transposed (Bt [NCOL][K]): within each group of
// 32 k, lane group lr takes k0 + 8 lr + s (s = 0..7), a permutation of the
// contraction index under which a lane's eight A values and eight B values
// are consecutive floats, loaded 16 bytes at a time.  The k loop is unrolled
// in full with the loads software-pipelined: the B fragments of group g + 2
// (from global memory, one L2 round trip) and the A fragments of group g + 1
// (from LDS) are issued before the 16 x WRB x WCB products of group g, in
// register sets of their own, so no product waits on a load issued just
// before it.
// Offset of B^T element (n, k): a plain [NCOL][K] array (P == 0), or a weight
// tensor W[K / P][NCOL][P] read in place (k = m P + p), where every run of 8
// consecutive k starting at a multiple of 8 stays within one m (P % 8 == 0).
template <int K, int NCOL, int P>
__device__ __forceinline__ int64_t bt_offset(int n, int k) {
    if constexpr (P == 0) {
        return (int64_t)n * K + k;
    } else {
        static_assert(P % 8 == 0 && K % P == 0, "runs of 8 k within one block of W");
        return ((int64_t)(k / P) * NCOL + n) * P + k % P;
    }
}

template <int K, int WCB, int NCBW, int NCOL = 0, int P = 0>
__device__ __forceinline__ void load_bt_f32(const float *__restrict__ Bt, int k0, int wc, int lr,
                                            int lc, float4 (&b)[2][WCB]) {
#pragma unroll
    for (int t = 0; t < WCB; ++t) {
        const float *p = Bt + bt_offset<K, NCOL, P>(16 * (wc + NCBW * t) + lc, k0 + 8 * lr);
        b[0][t] = *reinterpret_cast<const float4 *>(p);
        b[1][t] = *reinterpret_cast<const float4 *>(p + 4);
    }
}

template <int S, int WRB, int NRG>
__device__ __forceinline__ void load_a_f32(const float *As, int k0, int wr, int lr, int lc,
                                           float4 (&a)[WRB][2]) {
#pragma unroll
    for (int u = 0; u < WRB; ++u) {
        const float *p = As + (16 * (wr + NRG * u) + lc) * S + k0 + 8 * lr;
        a[u][0] = *reinterpret_cast<const float4 *>(p);
        a[u][1] = *reinterpret_cast<const float4 *>(p + 4);
    }
}

template <int WRB, int WCB>
__device__ __forceinline__ void mma_group_f32t(const float4 (&a)[WRB][2],
                                               const float4 (&b)[2][WCB],
                                               floatx4 (&acc)[WRB][WCB]) {
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int u = 0; u < WRB; ++u)
#pragma unroll
                for (int t = 0; t < WCB; ++t)
                    acc[u][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[u][h][q], b[h][t][q],
                                                                      acc[u][t], 0, 0, 0);
}

template <int K, int S, int WRB, int WCB, int NCBW, int NRG, int NCOL = 0, int P = 0>
__device__ __forceinline__ void mfma_lds_x_global_f32t(const float *As,
                                                       const float *__restrict__ Bt, int wr,
                                                       int wc, floatx4 (&acc)[WRB][WCB]) {
    constexpr int KG = 32;
    constexpr int NG = K / KG;
    static_assert(K % KG == 0 && NG >= 2, "K must be a multiple of 32, at least 64");
    const int lane = threadIdx.x & 63;
    const int lr = lane >> 4, lc = lane & 15;
    float4 b[3][2][WCB];
    float4 a[2][WRB][2];
    load_bt_f32<K, WCB, NCBW, NCOL, P>(Bt, 0, wc, lr, lc, b[0]);
    load_bt_f32<K, WCB, NCBW, NCOL, P>(Bt, KG, wc, lr, lc, b[1]);
    load_a_f32<S, WRB, NRG>(As, 0, wr, lr, lc, a[0]);
#pragma unroll
    for (int g = 0; g < NG; ++g) {
        if (g + 2 < NG)
            load_bt_f32<K, WCB, NCBW, NCOL, P>(Bt, (g + 2) * KG, wc, lr, lc, b[(g + 2) % 3]);
        if (g + 1 < NG) load_a_f32<S, WRB, NRG>(As, (g + 1) * KG, wr, lr, lc, a[(g + 1) % 2]);
        __builtin_amdgcn_sched_barrier(0);
        mma_group_f32t<WRB, WCB>(a[g % 2], b[g % 3], acc);
        __builtin_amdgcn_sched_barrier(0);
    }
}

template <int K, int WCB, int NCBW, int NCOL = 0, int P = 0>
__device__ __forceinline__ void load_b_bf16(const uint16_t *__restrict__ Bt, int k0, int wc,
                                            int lk, int lc, bf16x8 (&b)[4][WCB]) {
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int t = 0; t < WCB; ++t)
            b[s][t] = *reinterpret_cast<const bf16x8 *>(
                Bt + bt_offset<K, NCOL, P>(16 * (wc + NCBW * t) + lc, k0 + 32 * s + lk));
}

template <int S, int WRB, int WCB, int NRG>
__device__ __forceinline__ void mma_group_bf16(const uint16_t *As, int k0, int wr, int lk, int lc,
                                               const bf16x8 (&b)[4][WCB],
                                               floatx4 (&acc)[WRB][WCB]) {
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
                acc[u][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[u], b[s][t], acc[u][t], 0, 0, 0);
    }
}

template <int K, int S, int WRB, int WCB, int NCBW, int NRG, int NCOL = 0, int P = 0>
__device__ __forceinline__ void mfma_lds_x_global_bf16(const uint16_t *As,
                                                       const uint16_t *__restrict__ Bt, int wr,
                                                       int wc, floatx4 (&acc)[WRB][WCB]) {
    constexpr int KG = 128;  // 4 MFMA k-steps of 32
    static_assert(K % (2 * KG) == 0, "K must be a multiple of 256");
    const int lane = threadIdx.x & 63;
    const int lk = 8 * (lane >> 4), lc = lane & 15;
    bf16x8 b0[4][WCB], b1[4][WCB];
    load_b_bf16<K, WCB, NCBW, NCOL, P>(Bt, 0, wc, lk, lc, b0);
#pragma unroll 1
    for (int k0 = 0; k0 < K; k0 += 2 * KG) {
        load_b_bf16<K, WCB, NCBW, NCOL, P>(Bt, k0 + KG, wc, lk, lc, b1);
        __builtin_amdgcn_sched_barrier(0);
        mma_group_bf16<S, WRB, WCB, NRG>(As, k0, wr, lk, lc, b0, acc);
        const int kn = k0 + 2 * KG < K ? k0 + 2 * KG : K - KG;
        load_b_bf16<K, WCB, NCBW, NCOL, P>(Bt, kn, wc, lk, lc, b0);
        __builtin_amdgcn_sched_barrier(0);
        mma_group_bf16<S, WRB, WCB, NRG>(As, k0 + KG, wr, lk, lc, b1, acc);
    }
}

// Tile rows per block: 64 while the G tile fits 64 KiB; else 32, or 16 for
// wide outputs (128 and more channels), where a block's contraction is long
// enough that three smaller blocks per CU overlap gathers and contractions
// better than two larger ones (measured: C_out 128 fp32 36 -> 32 us; C_out 64
// fp32 stays at 32 rows, 42 -> 49 us with 16).
constexpr int fwd_tile_rows(int K, int CO, bool bf) {
    return (K * (bf ? 2 : 4) * 64 <= 65536) ? 64 : (CO >= 128 ? 16 : 32);
}

// Logical tile of physical block b of n: consecutive blocks are dispatched to
// the 8 XCDs in turn, so this gives each XCD one contiguous range of tiles and
// keeps the rows an XCD gathers local to its L2.
__device__ __forceinline__ int32_t xcd_tile(int32_t b, int32_t n) {
    const int32_t per = n / 8, rem = n % 8;
    const int32_t x = b % 8, l = b / 8;
    return x < rem ? x * (per + 1) + l : rem * (per + 1) + (x - rem) * per + l;
}

// First tile of XCD x's range when the persistent kernels split n_tiles tiles
// of TR rows over X XCDs: the ranges hold equal shares of the work estimate
// (edges + kRowCost per row, from the pattern's pointer array), so an XCD
// whose part of a bursty stream is dense gets fewer tiles.  Every block of
// the range still takes a fixed set of its tiles, so results do not depend
// on timing.
constexpr int64_t kRowCost = 8;

// quant: the workers (blocks or waves) that share an XCD's range.  When the
// tiles divide evenly among all workers, the ranges are rounded to multiples
// of quant, so every worker keeps the same number of tiles (a tile more for
// some would cost the kernel a whole tile's time).
__device__ __forceinline__ int32_t xcd_range_begin(int32_t x, int32_t X, int32_t n_tiles, int TR,
                                                   const int32_t *__restrict__ ptr,
                                                   int32_t n_rows, int32_t nnz, int32_t quant) {
    if (x <= 0) return 0;
    if (x >= X) return n_tiles;
    auto work = [&](int32_t t) {  // work estimate of the rows before tile t
        int32_t r = t * TR;
        r = r < n_rows ? r : n_rows;
        int32_t e = ptr[r];
        e = e < 0 ? 0 : (e < nnz ? e : nnz);
        return (int64_t)e + kRowCost * r;
    };
    const int64_t target = (work(n_tiles) * x) / X;
    if (target <= 0) return 0;
    // the first tile t with work(t) >= target, in (lo, hi]: each round the 64
    // lanes of the wave probe 64 points of the interval (work(0) = 0 < target)
    const int lane = threadIdx.x & 63;
    int32_t lo = 0, hi = n_tiles;
    while (hi - lo > 1) {
        const int64_t span = hi - lo;
        const int32_t t = lo + (int32_t)(((lane + 1) * span + 63) / 64);
        const uint64_t ge = __ballot(work(t) >= target);  // lane 63 probes hi: always set
        const int f = __builtin_ctzll(ge);
        const int32_t nhi = lo + (int32_t)(((f + 1) * span + 63) / 64);
        const int32_t nlo = f == 0 ? lo : lo + (int32_t)((f * span + 63) / 64);
        lo = nlo;
        hi = nhi;
    }
    if (quant > 0 && n_tiles % ((int64_t)X * quant) == 0) {
        const int32_t r = (hi + quant / 2) / quant * quant;
        return r < n_tiles ? r : n_tiles;
    }
    return hi;
}

// ================================================================ forward
constexpr int kFwdWaves = 4;

template <int M, int CI, int CO, int kBasis, bool kBf>
__global__ void __launch_bounds__(kFwdWaves * 64, fwd_tile_rows(M * CI, CO, kBf) == 16 ? 3 : 2)
    fwd_fused_kernel(int32_t n_out, const int32_t *__restrict__ row_ptr,
                     const int32_t *__restrict__ col_idx, const float *__restrict__ v,
                     KGeo g, const void *__restrict__ F, const void *__restrict__ Wop,
                     float *__restrict__ Y) {
    constexpr int NW = kFwdWaves;
    constexpr int K = M * CI;
    constexpr int TR = fwd_tile_rows(K, CO, kBf);
    constexpr int S = K + (kBf ? 8 : 4);           // padded LDS row (elements)
    constexpr int NRB = TR / 16, NCB = CO / 16;
    static_assert(CO % 16 == 0 && CI % 4 == 0, "shape");
    constexpr int NCBW = NCB < NW ? NCB : NW;      // column groups of waves
    constexpr int NRG = NW / NCBW;                 // row groups of waves
    static_assert(NCB % NCBW == 0 && NRB % NRG == 0, "tile split");
    constexpr int WCB = NCB / NCBW, WRB = NRB / NRG;
    constexpr int RPW = TR / NW;

    using GT = typename std::conditional<kBf, uint16_t, float>::type;
    __shared__ __attribute__((aligned(16))) GT Gs[TR * S];
    __shared__ EdgeStage<M> stage[NW];

    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const int32_t row0 = xcd_tile(blockIdx.x, gridDim.x) * TR;
    const double inv_r = g.inv_r;
    const float inv_tau = g.inv_tau;

    gather_rows<M, CI, kBasis, kBf, kBf, false, RPW, false>(
        row0 + w * RPW, n_out, row_ptr, col_idx, nullptr, v, g, F, Gs, S, w * RPW, stage[w],
        inv_r, inv_tau,
        GatherAhead{load_bound<RPW>(row_ptr, n_out, row0 + w * RPW, g.nnz), 0, false},
        -1);
    __syncthreads();

    const int wc = w % NCBW, wr = w / NCBW;
    floatx4 acc[WRB][WCB];
#pragma unroll
    for (int u = 0; u < WRB; ++u)
#pragma unroll
        for (int t = 0; t < WCB; ++t) acc[u][t] = floatx4{0.f, 0.f, 0.f, 0.f};

    if constexpr (!kBf)
        mfma_lds_x_global_f32t<K, S, WRB, WCB, NCBW, NRG>(
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

// ================================================================ row order
// The register-resident forward runs a tile's 16 rows in step, as long as its
// longest row.  Rows are ordered by length within windows of kOrderWindow
// consecutive rows (longest first, ties by index): a tile then holds rows of
// similar length, while a window stays a short stretch of the pattern (the
// rows an XCD gathers stay local to its L2).  order[p] is the row at
// position p; each row's result is the same whatever tile it is in.
// A wave sorts a window in registers (four rows a lane, a bitonic network
// whose cross-lane steps are lane shuffles).
constexpr int kOrderWindow = 256;
constexpr int kOrderThreads = 256;  // a window per wave

__global__ void __launch_bounds__(kOrderThreads)
    row_order_kernel(int32_t n_rows, const int32_t *__restrict__ ptr, int32_t nnz,
                     int32_t *__restrict__ order) {
    const int lane = threadIdx.x & 63;
    const int32_t win = blockIdx.x * (kOrderThreads / 64) + (threadIdx.x >> 6);
    const int32_t r0 = win * kOrderWindow;
    if (r0 >= n_rows) return;
    // key: (longest first) length complement above the index in the window;
    // positions past the last row sort behind every row
    uint32_t k[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int32_t r = r0 + 4 * lane + j;
        k[j] = 0xFFFFFFFFu;
        if (r < n_rows) {
            int32_t a = ptr[r], b = ptr[r + 1];
            a = a < 0 ? 0 : (a < nnz ? a : nnz);
            b = b < a ? a : (b < nnz ? b : nnz);
            const uint32_t len = (uint32_t)(b - a) < 0xFFFFFFu ? (uint32_t)(b - a) : 0xFFFFFFu;
            k[j] = ((0xFFFFFFu - len) << 8) | (uint32_t)(4 * lane + j);
        }
    }
    // bitonic sort, ascending, of element i = 4 lane + j
#pragma unroll
    for (int size = 2; size <= kOrderWindow; size <<= 1) {
#pragma unroll
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            if (stride >= 4) {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const uint32_t o = __shfl_xor(k[j], stride >> 2, 64);
                    const int i = 4 * lane + j;
                    const bool asc = (i & size) == 0, lower = (i & stride) == 0;
                    k[j] = (asc == lower) ? (k[j] < o ? k[j] : o) : (k[j] > o ? k[j] : o);
                }
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    if (j & stride) continue;
                    const int i = 4 * lane + j;
                    const bool asc = (i & size) == 0;
                    const uint32_t x = k[j], y = k[j | stride];
                    if ((x > y) == asc) {
                        k[j] = y;
                        k[j | stride] = x;
                    }
                }
            }
        }
    }
    // The persistent forward hands each wave tiles a fixed stride apart, often a
    // multiple of a window's tiles, so a wave would sit at the same place in
    // every window: a full window's tiles are rotated by a hash of its index
    // (the last, partial window keeps its rows in front).  Position q = 4 lane
    // + j takes sorted element ((q / 16 + rot) % 16) * 16 + q % 16, which has
    // the same j.
    constexpr int kTiles = kOrderWindow / 16;
    const bool full = r0 + kOrderWindow <= n_rows;
    const uint32_t rot = full ? ((uint32_t)win * 2654435761u) >> 28 : 0u;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int q = 4 * lane + j;
        const int src = (int)(((uint32_t)(q / 16) + rot) % kTiles) * 16 + q % 16;
        const uint32_t key = __shfl(k[j], src >> 2, 64);
        if (r0 + q < n_rows) order[r0 + q] = r0 + (int32_t)(key & 255u);
    }
}

// ================================================================ forward, G in registers
// Each wave owns tiles of 16 output rows: lane l serves row (l & 15) and
// channel group g = l >> 4, i.e. channels [g*CI/4, (g+1)*CI/4) of every basis
// function.  G accumulates in registers and is the MFMA A operand as is: at
// k-step s lane group g contributes G[row, m(s), g*CI/4 + t(s)], so the
// contraction index is a permutation of (m, c) that the W operand follows.
// W sits in LDS, staged once per persistent block; waves then run their
// tiles independently, so one wave's gather overlaps another's MFMAs.
constexpr int kRegWaves = 8;

// bytes of W in LDS for the register-resident forward
template <int M, int CI, int CO, bool kBf>
constexpr int reg_w_bytes() {
    return M * CI * CO * (kBf ? 2 : 4) + (kBf ? CO * 16 : 0);
}

template <int M, int CI, int CO, bool kBf>
constexpr bool reg_forward_fits() {
    // float32 rows wider than 32 channels hold M*CI/4 gather accumulators per
    // lane and spend long on float32 MFMAs with two waves per SIMD; there the
    // LDS-tile kernel is faster.  bf16 rows of 64 channels still gain.
    return reg_w_bytes<M, CI, CO, kBf>() <= 131072 && CI % 16 == 0 &&
           (CI <= 32 || (kBf && CI <= 64)) && CO % 16 == 0 && (!kBf || (CI / 4) % 8 == 0);
}

// Waves per SIMD the register-resident forward is compiled for: four while
// the gather accumulators (M * CI / 4 per lane) leave room, else two.
template <int M, int CI>
constexpr int reg_waves_per_eu() {
    return M * CI / 4 <= 64 ? 4 : 2;
}

template <int M, int CI, int CO, int kBasis, bool kBf>
__global__ void __launch_bounds__(kRegWaves * 64)
    __attribute__((amdgpu_waves_per_eu(reg_waves_per_eu<M, CI>())))
    fwd_reg_kernel(int32_t n_out, int32_t n_tiles, const int32_t *__restrict__ row_ptr,
                   const int32_t *__restrict__ col_idx, const float *__restrict__ v,
                   KGeo g, const void *__restrict__ Fv, const void *__restrict__ Wv,
                   float *__restrict__ Y, const int32_t *__restrict__ order) {
    constexpr int K = M * CI;
    constexpr int CG = CI / 4;          // channels per lane group
    constexpr int NCB = CO / 16;        // 16-column blocks of Y
    constexpr int NT = kRegWaves * 64;
    static_assert(reg_forward_fits<M, CI, CO, kBf>(), "shape");
    // W in LDS.  float32: [K][16][NCB] (b for all column blocks of one (k, n)
    // contiguous);  bf16: [NCB][16][K + 8] (8 consecutive k of one n contiguous)
    constexpr int SWB = K + 8;
    constexpr int WLDS = kBf ? NCB * 16 * SWB * 2 : K * CO * 4;
    __shared__ __attribute__((aligned(16))) char Wl[WLDS];

    if constexpr (!kBf) {
        const float *W = static_cast<const float *>(Wv);  // [K, CO]
        float *Wf = reinterpret_cast<float *>(Wl);
        for (int q = threadIdx.x; q < K * CO; q += NT) {
            const int k = q / CO, n = q % CO;
            Wf[(k * 16 + (n & 15)) * NCB + (n >> 4)] = W[q];
        }
    } else {
        const uint16_t *W = static_cast<const uint16_t *>(Wv);  // [K, CO] bf16
        uint16_t *Wb = reinterpret_cast<uint16_t *>(Wl);
        for (int q = threadIdx.x; q < K * CO; q += NT) {
            const int k = q / CO, n = q % CO;
            Wb[((n >> 4) * 16 + (n & 15)) * SWB + k] = W[q];
        }
    }
    __syncthreads();

    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const int rl = lane & 15;        // row within the tile
    const int gq = lane >> 4;        // channel group
    const double inv_r = g.inv_r;
    const float inv_tau = g.inv_tau;

    // tiles of this wave: the block's XCD owns a contiguous range, its waves
    // interleave (with fewer than 8 blocks, one range per block)
    const int32_t G = gridDim.x, X = G < 8 ? G : 8;
    const int32_t x = blockIdx.x % X;
    const int32_t gx = G / X + (x < G % X ? 1 : 0);
    const int32_t waves_x = gx * kRegWaves;
    const int32_t lw = (blockIdx.x / X) * kRegWaves + w;
    // (rounding needs the same worker count on every XCD: the ranges' shared ends
    // are computed on both sides)
    const int32_t quant = G % X == 0 ? waves_x : 0;
    const int32_t t_begin = xcd_range_begin(x, X, n_tiles, 16, row_ptr, n_out, g.nnz, quant);
    const int32_t t_end = xcd_range_begin(x + 1, X, n_tiles, 16, row_ptr, n_out, g.nnz, quant);

#pragma unroll 1
    for (int32_t tile = t_begin + lw; tile < t_end; tile += waves_x) {
        // the tile's rows: positions tile*16 .. tile*16+15 of the row order
        const int32_t row = tile * 16 + rl < n_out ? order[tile * 16 + rl] : n_out;
        int32_t e0 = 0, e1 = 0;
        if (row < n_out) {
            e0 = row_ptr[row];
            e1 = row_ptr[row + 1];
            e0 = e0 < 0 ? 0 : (e0 < g.nnz ? e0 : g.nnz);
            e1 = e1 < e0 ? e0 : (e1 < g.nnz ? e1 : g.nnz);
        }
        int32_t len = e1 - e0;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int32_t o = __shfl_xor(len, d, 64);
            len = o > len ? o : len;
        }
        float acc[M][CG];
#pragma unroll
        for (int m = 0; m < M; ++m)
#pragma unroll
            for (int t = 0; t < CG; ++t) acc[m][t] = 0.f;

        // Four edges of the row per step, one per lane of the row's group:
        // lane gq loads the neighbour index of edge q + gq one step ahead and
        // evaluates that edge's basis; the group shares indices and basis
        // values through cross-lane reads, and every lane loads its channels
        // of all four neighbours' features.
        int32_t jn = (e0 + gq < e1) ? col_idx[e0 + gq] : 0;
#pragma unroll 1
        for (int32_t q = 0; q < len; q += 4) {
            const int32_t eo = e0 + q + gq;          // this lane's edge
            const int32_t jo = jn;
            jn = (eo + 4 < e1) ? col_idx[eo + 4] : 0;
            // features of the four edges, SB at a time (fewer registers for wide rows)
            constexpr int SB = CG <= 8 ? 4 : 2;
            float bo[M];
            bool have_basis = false;
#pragma unroll
            for (int u0 = 0; u0 < 4; u0 += SB) {
            float f[SB][CG];
#pragma unroll
            for (int us = 0; us < SB; ++us) {
                const int u = u0 + us;
                const int32_t j = __shfl(jo, rl + 16 * u, 64);
                if constexpr (kBf) {
                    const uint16_t *src = static_cast<const uint16_t *>(Fv) + (int64_t)j * CI + gq * CG;
#pragma unroll
                    for (int c = 0; c < CG; c += 8) {
                        const uint4 raw = *reinterpret_cast<const uint4 *>(src + c);
                        const uint32_t w4[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
                        for (int k = 0; k < 4; ++k) {
                            f[us][c + 2 * k] = __uint_as_float(w4[k] << 16);
                            f[us][c + 2 * k + 1] = __uint_as_float(w4[k] & 0xFFFF0000u);
                        }
                    }
                } else {
                    const float *src = static_cast<const float *>(Fv) + (int64_t)j * CI + gq * CG;
#pragma unroll
                    for (int c = 0; c < CG; c += 4) {
                        const float4 raw = *reinterpret_cast<const float4 *>(src + c);
                        f[us][c] = raw.x;
                        f[us][c + 1] = raw.y;
                        f[us][c + 2] = raw.z;
                        f[us][c + 3] = raw.w;
                    }
                }
            }
            // this lane's edge basis, once per step (zero past the row's end:
            // those lanes loaded row 0's features, which then carry no weight)
            if (!have_basis) {
                have_basis = true;
                if (eo < e1) {
                    edge_basis<M, kBasis>(g, v, row, jo, eo, inv_r, inv_tau, bo);
                } else {
#pragma unroll
                    for (int m = 0; m < M; ++m) bo[m] = 0.f;
                }
            }
#pragma unroll
            for (int us = 0; us < SB; ++us)
#pragma unroll
                for (int m = 0; m < M; ++m) {
                    const float bm = __shfl(bo[m], rl + 16 * (u0 + us), 64);
#pragma unroll
                    for (int t = 0; t < CG; ++t) acc[m][t] += bm * f[us][t];
                }
            }
        }

        // ---- Y rows of the tile = G W on the matrix cores
        floatx4 ay[NCB];
#pragma unroll
        for (int nb = 0; nb < NCB; ++nb) ay[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
        if constexpr (!kBf) {
            const float *Wf = reinterpret_cast<const float *>(Wl);
#pragma unroll
            for (int m = 0; m < M; ++m)
#pragma unroll
                for (int t = 0; t < CG; ++t) {
                    const int kB = m * CI + gq * CG + t;
                    float b[NCB];
#pragma unroll
                    for (int nb = 0; nb < NCB; ++nb) b[nb] = Wf[(kB * 16 + rl) * NCB + nb];
#pragma unroll
                    for (int nb = 0; nb < NCB; ++nb)
                        ay[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(acc[m][t], b[nb], ay[nb], 0, 0, 0);
                    if ((t & 3) == 3) __builtin_amdgcn_sched_barrier(0);
                }
        } else {
            const uint16_t *Wb = reinterpret_cast<const uint16_t *>(Wl);
#pragma unroll
            for (int m = 0; m < M; ++m)
#pragma unroll
                for (int t0 = 0; t0 < CG; t0 += 8) {
                    bf16x8 a;
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        const uint16_t hb = f2bf(acc[m][t0 + j]);
                        a[j] = __builtin_bit_cast(__bf16, hb);
                    }
                    const int kB = m * CI + gq * CG + t0;
#pragma unroll
                    for (int nb = 0; nb < NCB; ++nb) {
                        const bf16x8 b = *reinterpret_cast<const bf16x8 *>(&Wb[(nb * 16 + rl) * SWB + kB]);
                        ay[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, ay[nb], 0, 0, 0);
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
        }
        // D layout: lane holds tile rows 4*(l >> 4) + r, column l & 15 of each
        // block; lane 4 g + r (row 4 g + r of the tile) knows that row's index
        int32_t yrow[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) yrow[r] = __shfl(row, 4 * gq + r, 64);
#pragma unroll
        for (int nb = 0; nb < NCB; ++nb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int32_t yr = yrow[r];
                if (yr < n_out) Y[(int64_t)yr * CO + 16 * nb + rl] = ay[nb][r];
            }
    }
}

// ---------------------------------------------------------------- one-hot event forward
// The fixed-decay event basis gives an edge a single nonzero value, at its
// offset index k (none for the centre pixel), so of the M x CG products per
// edge and lane of the register forward, CG carry the sum.  A register cannot
// be chosen by a per-lane index, an LDS address can: here each lane keeps the
// G values it owns (4 channels of two tile rows, all 8 offsets) in a
// lane-private LDS slot, and an edge adds its 4 products per row into the
// slot of its offset, a read, 4 FMAs and a write.  Lanes write only their
// own slot, so no barrier is needed; LDS accesses of one wave complete in
// order, so consecutive edges of one offset chain correctly.  Per step the 4
// lanes of a row take 4 edges in pattern order, one each (index,
// coordinates, offset and decay), and share index, offset and weight by
// cross-lane reads; each lane adds its piece of the neighbour rows.  The
// next step's rows and coordinates are loaded while this step is summed, and
// the indices two steps ahead, across tiles.  Then Y rows = G W on the matrix
// cores, W in LDS as in the register forward.  The per-(row, offset, channel)
// sums take their edges in pattern order, as in the register forward.
constexpr int kOhWaves = 8;

template <int CI, int CO>
constexpr bool onehot_forward_fits() {
    return CI == 32 && CO % 16 == 0 &&
           8 * CI * CO * 4 + kOhWaves * 8 * CI * 16 * 4 <= 163840;
}

template <int CI, int CO>
__global__ void __launch_bounds__(kOhWaves * 64, 1)
    fwd_onehot_kernel(int32_t n_out, int32_t n_tiles, const int32_t *__restrict__ row_ptr,
                      const int32_t *__restrict__ col_idx, KGeo g, const float *__restrict__ F,
                      const float *__restrict__ W, float *__restrict__ Y,
                      const int32_t *__restrict__ order) {
    constexpr int M = 8;
    constexpr int K = M * CI;
    constexpr int CG = CI / 4;    // channels of a tile row per lane in the products
    constexpr int NCB = CO / 16;  // 16-column blocks of Y
    constexpr int NT = kOhWaves * 64;
    static_assert(onehot_forward_fits<CI, CO>(), "shape");
    __shared__ __attribute__((aligned(16))) float Wf[K * CO];  // [K][16][NCB]
    // G of a wave: [offset k][half h][position], 16 bytes each (below)
    __shared__ float4 Gs[kOhWaves][2 * M][64];

    for (int q = threadIdx.x; q < K * CO; q += NT) {
        const int k = q / CO, n = q % CO;
        Wf[(k * 16 + (n & 15)) * NCB + (n >> 4)] = W[q];
    }
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    // Two roles per lane.  As a basis lane it takes edge gq of each step of
    // tile row rl: index, coordinates, offset and decay.  As a sum lane it
    // loads piece pc (16 bytes, 4 channels) of the neighbour rows of tile
    // rows r8 and r8 + 8, so one load instruction takes 8 whole rows, and
    // keeps the G values of those two rows and 4 channels for all offsets.
    // The 16 bytes of sum lane L sit at position L ^ (L / 8 mod 8), which
    // keeps both its own accesses and the products' reads (lanes 8 apart)
    // on distinct banks.
    const int rl = lane & 15;  // basis lane: row within the tile
    const int gq = lane >> 4;  //             edge of the step
    const int r8 = lane >> 3;  // sum lane: tile rows r8, r8 + 8
    const int pc = lane & 7;   //           piece of the row
    auto pos = [](int L) { return L ^ ((L >> 3) & 7); };
    float4 *gl = &Gs[w][0][pos(lane)];
#pragma unroll
    for (int p = 0; p < 2 * M; ++p) gl[64 * p] = make_float4(0.f, 0.f, 0.f, 0.f);
    __syncthreads();

    const float inv_tau = g.inv_tau;
    const int32_t nnz = g.nnz;
    const int32_t G = gridDim.x, X = G < 8 ? G : 8;
    const int32_t x = blockIdx.x % X;
    const int32_t gx = G / X + (x < G % X ? 1 : 0);
    const int32_t waves_x = gx * kOhWaves;
    const int32_t lw = (blockIdx.x / X) * kOhWaves + w;
    const int32_t quant = G % X == 0 ? waves_x : 0;
    const int32_t t_begin = xcd_range_begin(x, X, n_tiles, 16, row_ptr, n_out, nnz, quant);
    const int32_t t_end = xcd_range_begin(x + 1, X, n_tiles, 16, row_ptr, n_out, nnz, quant);

    // Loads take 32-bit byte offsets from the arrays' bases: the host takes
    // this kernel while F, the packed events and the pattern are under 4 GiB
    // (so rows and tiles are far below 2^31), and only with nnz >= 1.  Index
    // loads read positions clamped into [0, nnz) and use the value only
    // inside the row; past its end an edge weighs 0 and reads row 0.
    const char *Fb = reinterpret_cast<const char *>(F);
    const char *Eb = reinterpret_cast<const char *>(g.ev);
    const char *Ib = reinterpret_cast<const char *>(col_idx);
    const uint32_t fo = (uint32_t)(pc * 16);  // the sum lane's piece
    auto idx_raw = [&](int32_t e) {
        const uint32_t c = (uint32_t)(e < nnz ? e : nnz - 1);
        return *reinterpret_cast<const int32_t *>(Ib + (c << 2));
    };
    auto ev_at = [&](int32_t r) {
        return *reinterpret_cast<const int4 *>(Eb + ((uint32_t)r << 4));
    };
    // j: the basis lane's neighbour; f[u][h]: the sum lane's piece of the
    // neighbour of edge u of tile row r8 + 8 h
    auto load_step = [&](int32_t j, int4 &ev, float4 (&f)[4][2]) {
        ev = ev_at(j);
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const uint32_t ju = (uint32_t)__shfl(j, r8 + 8 * h + 16 * u, 64);
                f[u][h] = *reinterpret_cast<const float4 *>(Fb + (ju * (uint32_t)(CI * 4) + fo));
            }
    };
    // a tile's row of this lane: loaded at a clamped position, replaced by
    // n_out past the wave's tiles or the rows
    auto order_raw = [&](int32_t t) {
        const int32_t q = t * 16 + rl;
        return order[q < n_out ? q : n_out - 1];
    };
    auto row_of = [&](int32_t t, int32_t raw) {
        return t < t_end && t * 16 + rl < n_out ? raw : n_out;
    };
    auto bounds_raw = [&](int32_t r, int32_t &b0, int32_t &b1) {
        const int32_t q = r < n_out ? r : n_out - 1;
        b0 = row_ptr[q];
        b1 = row_ptr[q + 1];
    };
    auto clamp_bounds = [&](int32_t r, int32_t b0, int32_t b1, int32_t &e0, int32_t &e1) {
        b0 = b0 < 0 ? 0 : (b0 < nnz ? b0 : nnz);
        b1 = b1 < b0 ? b0 : (b1 < nnz ? b1 : nnz);
        e0 = r < n_out ? b0 : 0;
        e1 = r < n_out ? b1 : 0;
    };
    auto wave_steps = [&](int32_t e0, int32_t e1) {  // steps of 4 edges of the longest row
        int32_t len = e1 - e0;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int32_t o = __shfl_xor(len, d, 64);
            len = o > len ? o : len;
        }
        return __builtin_amdgcn_readfirstlane((len + 3) >> 2);
    };

    int32_t tile = t_begin + lw;
    if (tile >= t_end) return;  // (wave-uniform; no barrier follows)
    // The tile pipeline: at the start of tile t the bounds of tile t + 1 are
    // there (loaded at the start of t - 1) and the rows of t + 2; its
    // coordinates, the bounds of t + 2 and the rows of t + 3 are loaded then.
    int32_t row = row_of(tile, order_raw(tile));
    int32_t row_n = row_of(tile + waves_x, order_raw(tile + waves_x));
    int32_t row_nn_raw = order_raw(tile + 2 * waves_x);
    int32_t e0, e1, b0n, b1n;
    {
        int32_t b0, b1;
        bounds_raw(row, b0, b1);
        clamp_bounds(row, b0, b1, e0, e1);
    }
    bounds_raw(row_n, b0n, b1n);
    int4 a = ev_at(row < n_out ? row : 0);
    int32_t steps = wave_steps(e0, e1);
    int32_t jx = idx_raw(e0 + gq);
    int32_t jy = idx_raw(e0 + 4 + gq);
    int4 eva, evb;
    float4 fa[4][2], fb[4][2];
    load_step(e0 + gq < e1 ? jx : 0, eva, fa);

    // The edge of this lane in a step: offset and decay (weight 0 past the
    // row's end and for the centre pixel), shared with the row's lanes, and
    // the sums of the step's four edges into their slots.
    auto sum_step = [&](int32_t e, const int4 &ev, const float4 (&f)[4][2]) {
        int k = event_index(a.x - ev.x, a.y - ev.y);
        float d = event_decay(a.z, ev.z, inv_tau);
        const bool live = e < e1 && k >= 0;
        k = live ? k : 0;
        d = live ? d : 0.f;
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int ku = __shfl(k, r8 + 8 * h + 16 * u, 64);
                const float du = __shfl(d, r8 + 8 * h + 16 * u, 64);
                float4 *sl = gl + 64 * (2 * ku + h);
                float4 acc = *sl;
                acc.x = fmaf(du, f[u][h].x, acc.x);
                acc.y = fmaf(du, f[u][h].y, acc.y);
                acc.z = fmaf(du, f[u][h].z, acc.z);
                acc.w = fmaf(du, f[u][h].w, acc.w);
                *sl = acc;
            }
    };

#pragma unroll 1
    for (;;) {
        const int32_t tn = tile + waves_x;
        const int32_t row_nn = row_of(tn + waves_x, row_nn_raw);
        row_nn_raw = order_raw(tn + 2 * waves_x);
        int32_t e0n, e1n;
        clamp_bounds(row_n, b0n, b1n, e0n, e1n);
        bounds_raw(row_nn, b0n, b1n);
        const int4 an = ev_at(row_n < n_out ? row_n : 0);
        // Step s takes edges e0 + 4 s .. + 3 of each row.  Its indices are
        // loaded at step s - 2 and its rows and coordinates at s - 1, into
        // two register sets used in turn (a copy between them would wait for
        // the loads).  The steps of consecutive tiles form one stream: the
        // last pair of a tile loads the next tile's first steps, which land
        // while this tile's products run.  Every pair issues the same loads
        // (its second step is summed only if the tile has it), so the
        // compiler's waits stay those of one step ahead.
        int32_t e = e0 + gq;
        int32_t s = 0;
        do {
            const bool last = s + 2 >= steps;
            jx = idx_raw(last ? e0n + gq : e + 8);
            load_step(e + 4 < e1 ? jy : 0, evb, fb);
            __builtin_amdgcn_sched_barrier(0);  // the loads go out before the sums wait
            sum_step(e, eva, fa);
            e += 4;
            jy = idx_raw(last ? e0n + 4 + gq : e + 8);
            load_step((last ? e0n + gq < e1n : e + 4 < e1) ? jx : 0, eva, fa);
            __builtin_amdgcn_sched_barrier(0);
            if (s + 1 < steps) sum_step(e, evb, fb);
            e += 4;
            s += 2;
        } while (s < steps);

        // ---- Y rows of the tile = G W on the matrix cores; the slot is
        // cleared for the next tile as it is read
        floatx4 ay[NCB];
#pragma unroll
        for (int nb = 0; nb < NCB; ++nb) ay[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
        // lane (rl, gq) takes channels 8 gq .. 8 gq + 7 of tile row rl: pieces
        // 2 gq, 2 gq + 1 of the sum lanes of that row
        float4 *gr = &Gs[w][rl >> 3][0];
        const int pr0 = pos(8 * (rl & 7) + 2 * gq), pr1 = pos(8 * (rl & 7) + 2 * gq + 1);
#pragma unroll
        for (int m = 0; m < M; ++m) {
            float av[CG];
            const float4 v0 = gr[128 * m + pr0], v1 = gr[128 * m + pr1];
            av[0] = v0.x;
            av[1] = v0.y;
            av[2] = v0.z;
            av[3] = v0.w;
            av[4] = v1.x;
            av[5] = v1.y;
            av[6] = v1.z;
            av[7] = v1.w;
            gr[128 * m + pr0] = make_float4(0.f, 0.f, 0.f, 0.f);
            gr[128 * m + pr1] = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
            for (int t = 0; t < CG; ++t) {
                const int kB = m * CI + gq * CG + t;
                float b[NCB];
#pragma unroll
                for (int nb = 0; nb < NCB; ++nb) b[nb] = Wf[(kB * 16 + rl) * NCB + nb];
#pragma unroll
                for (int nb = 0; nb < NCB; ++nb)
                    ay[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[t], b[nb], ay[nb], 0, 0, 0);
                if ((t & 3) == 3) __builtin_amdgcn_sched_barrier(0);
            }
        }
        int32_t yrow[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) yrow[r] = __shfl(row, 4 * gq + r, 64);
#pragma unroll
        for (int nb = 0; nb < NCB; ++nb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int32_t yr = yrow[r];
                if (yr < n_out) Y[(int64_t)yr * CO + 16 * nb + rl] = ay[nb][r];
            }

        tile = tn;
        if (tile >= t_end) break;
        row = row_n;
        row_n = row_nn;
        a = an;
        e0 = e0n;
        e1 = e1n;
        steps = wave_steps(e0, e1);
    }
}

// ================================================================ backward, wave-specialised
// Persistent blocks over tiles of TR input rows, with the waves in two roles:
// NG gather waves build tile s+1 (D rows through the transposed pattern, and
// F rows) in one half of a double-buffered LDS tile while NM matrix waves run
// the matrix work of tile s on the other half (dF = D Wt, dW += F^T D); one
// block barrier per step hands the halves over, so the gathers' memory
// latency overlaps the matrix cores' work.  The matrix waves read Wt from
// memory or from registers (their slice, loaded once).
enum WLoc { kWGlobal = 0, kWRegs = 1 };

// Per shape: waves of each role, tile rows and where Wt lives, sized so that
// the registers allow all waves on one CU and the LDS tiles fit:
//   narrow float32 rows   8 + 4 waves, 32 rows, Wt slice in registers;
//   otherwise             4 + 4 waves, 32 rows, Wt slice in registers if it
//                         takes at most 64 of them, else from memory.
// (Measured on the 64-channel shapes: 8 + 8 waves with 16-row float32 tiles,
// or with Wt in LDS for bf16, ran slower than 4 + 4.)
struct WsCfg {
    int ng, nm, tr, wloc;
};

// Tile rows of the fixed-decay event backward on rows of 32 float32
// channels: its in-place gather keeps no stage in LDS, which leaves room for
// 64-row tiles (half the block barriers of 32-row ones)
constexpr int kEventRmwTR = 64;

template <int M, int CI, int CO, bool kBf>
constexpr WsCfg ws_cfg() {
    if (!kBf && CI <= 32 && CO <= 32)  // wider D rows (M*CO > 256) leave LDS for 4 gather waves
        return M * CO <= 256 ? WsCfg{8, 4, 32, kWRegs} : WsCfg{4, 4, 32, kWGlobal};
    // 16 columns of Wt per matrix wave (one dF column block), K2 = M*CO rows
    return WsCfg{4, 4, 32, (kBf ? M * CO <= 512 : M * CO <= 256) ? kWRegs : kWGlobal};
}

template <int M, int CI, int CO, int kBasis, bool kBf,
          int kWsGather = ws_cfg<M, CI, CO, kBf>().ng,
          int kWsMma = ws_cfg<M, CI, CO, kBf>().nm,
          int kTR = ws_cfg<M, CI, CO, kBf>().tr,
          int kWLoc = ws_cfg<M, CI, CO, kBf>().wloc, bool kAllowRmw = true>
__global__ void __launch_bounds__((kWsGather + kWsMma) * 64, 1)
    bwd_ws_kernel(int32_t n_in, int32_t n_tiles, const int32_t *__restrict__ col_ptr,
                  const int32_t *__restrict__ row_idx, const int32_t *__restrict__ perm,
                  const float *__restrict__ v, KGeo g, const void *__restrict__ Fv,
                  const void *__restrict__ dY, const void *__restrict__ Wop,
                  float *__restrict__ dF, float *__restrict__ dW_part) {
    // dF == nullptr: no input gradient; dW_part == nullptr: no weight gradient
    constexpr int TR = kTR;
    constexpr int K2 = M * CO;
    constexpr int SD = K2 + (kBf ? 8 : 4);
    constexpr int SF = CI + (kBf ? 8 : 4);
    constexpr int RPW = TR / kWsGather;
    static_assert(CI % 16 == 0 && CO % 16 == 0 && TR % kWsGather == 0, "shape");
    static_assert(!kBf || TR % 32 == 0, "bf16 dW takes 32 rows per MFMA k-step");
    // dF tile [TR, CI]: 16x16 blocks over the matrix waves
    constexpr int NRB = TR / 16, NCB = CI / 16;
    constexpr int NCBW = NCB < kWsMma ? NCB : kWsMma;
    constexpr int NRG_ = kWsMma / NCBW;
    constexpr int NRG = NRG_ < NRB ? NRG_ : NRB;  // waves past NCBW * NRG have no dF block
    static_assert(NCB % NCBW == 0 && NRB % NRG == 0, "dF split");
    constexpr int WCB = NCB / NCBW, WRB = NRB / NRG;
    // dW [CI, K2]: each matrix wave owns K2/NM columns, all CI rows
    constexpr int NWB = (K2 / 16) / kWsMma;
    constexpr int NIB = CI / 16;
    static_assert((K2 / 16) % kWsMma == 0, "dW split");

    using DT = typename std::conditional<kBf, uint16_t, float>::type;
    __shared__ __attribute__((aligned(16))) DT Ds[2][TR * SD];
    __shared__ __attribute__((aligned(16))) DT Fs[2][TR * SF];
    // the fixed-decay event basis takes the one-hot gather while its stage (a
    // chunk of 64 neighbour rows per gather wave) fits in LDS.  (Chunks of 32
    // leave the registers for four bucket rows read together, but a chunk
    // then spans about half of a wave's rows, and the walk ran slower.)
    constexpr int CK = 64;
    constexpr int RBY = CO * (int)sizeof(DT);  // bytes per gathered row
    constexpr bool kOneHotShape =
        kBasis == SBC_BASIS_EVENT8 + 1 && M == 8 && RPW * M <= 64 && 64 % (RPW * M) == 0 &&
        RBY % 16 == 0 && 64 % (RBY / 16) == 0 && CK % (64 / (RBY / 16)) == 0;
    // rows of 32 float32 channels, 4 or 8 per gather wave: the in-place
    // one-hot gather (no stage)
    // (also the learned decays and their derivatives, M / 8 values per edge)
    constexpr bool kDecayBasis =
        (kBasis == SBC_BASIS_EVENT_DECAYS + 1 || kBasis == kDecayDerivMode) && M % 8 == 0;
    constexpr bool kRmw = kAllowRmw && (kOneHotShape || kDecayBasis) && !kBf && CO == 32 &&
                          (RPW == 4 || RPW == 8) && 2 * TR * (SD + SF) * sizeof(DT) <= 163840;
    constexpr bool kOneHot =
        kOneHotShape &&
        (kRmw ||
         2 * TR * (SD + SF) * sizeof(DT) + kWsGather * sizeof(OneHotStage<RBY, CK>) <= 163840);
    struct NoStage {};
    using Stage = typename std::conditional<
        kRmw, NoStage,
        typename std::conditional<kOneHot, OneHotStage<RBY, CK>, EdgeStage<M>>::type>::type;
    __shared__ __attribute__((aligned(16))) Stage stage[kWsGather];

    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const bool gatherer = w < kWsGather;
    const int mw = w - kWsGather;
    const int wc = mw % NCBW, wr = mw / NCBW;
    const double inv_r = g.inv_r;
    const float inv_tau = g.inv_tau;

    // tiles of this block: its XCD's contiguous range, interleaved over the
    // XCD's blocks (with fewer than 8 blocks, one range per block)
    const int32_t G = gridDim.x, X = G < 8 ? G : 8;
    const int32_t x = blockIdx.x % X, l = blockIdx.x / X;
    const int32_t gx = G / X + (x < G % X ? 1 : 0);
    const int32_t quant = G % X == 0 ? gx : 0;  // the same on every XCD (shared range ends)
    const int32_t t_first = xcd_range_begin(x, X, n_tiles, TR, col_ptr, n_in, g.nnz, quant) + l;
    const int32_t t_end = xcd_range_begin(x + 1, X, n_tiles, TR, col_ptr, n_in, g.nnz, quant);
    const int32_t n_my = t_first < t_end ? (t_end - t_first + gx - 1) / gx : 0;

    // row bounds (and first neighbour indices) of the gather's next tile,
    // loaded one tile ahead; the one-hot gather keeps its own loads in flight
    // further ahead (OneHotPipe)
    GatherAhead ahead{
        n_my > 0 && !kOneHot ? load_bound<RPW>(col_ptr, n_in, t_first * TR + w * RPW, g.nnz) : 0,
        0, false};
    constexpr int NR = kOneHot ? CK / (64 / (RBY / 16)) : 1;  // row pieces per lane and chunk
    OneHotPipe<NR> pipe;
    using RG = RmwGather<32, kRmw ? RPW : 4, kRmw && kDecayBasis ? M / 8 : 1,
                         !(kRmw && kDecayBasis) ? 0 : (kBasis == kDecayDerivMode ? 2 : 1)>;
    const RG rmw{col_ptr, row_idx, g.ev, static_cast<const float *>(dY), g.decays, n_in, g.nnz,
                 inv_tau, lane / RG::LPR, lane % RG::LPR};
    typename RG::Pipe rpipe;
    auto wave_rows = [&](int32_t s) {
        return s < n_my ? (t_first + s * gx) * TR + w * RPW : -1;
    };
    auto load_tile = [&](int32_t s, int buf) {
        if constexpr (kRmw) {
            gather_rows_rmw(rmw, wave_rows(s + 2), wave_rows(s + 3),
                            reinterpret_cast<float *>(Ds[buf]), SD, w * RPW, rpipe);
        } else if constexpr (kOneHot) {
            const OneHotTiles tl{wave_rows(s), wave_rows(s + 1), wave_rows(s + 2),
                                 wave_rows(s + 3)};
            gather_rows_onehot<CO, RPW, true, kBf, NR>(tl, n_in, col_ptr, row_idx, g, dY,
                                                       Ds[buf], SD, w * RPW, stage[w], inv_tau,
                                                       pipe);
        } else {
            ahead = gather_rows<M, CO, kBasis, kBf, kBf, true, RPW, true>(
                wave_rows(s), n_in, col_ptr, row_idx, perm, v, g, dY, Ds[buf], SD, w * RPW,
                stage[w], inv_r, inv_tau, ahead, wave_rows(s + 1));
        }
    };

    // The two roles run separate loops (so the matrix waves' dW accumulators
    // are not live in the gather code); each role passes the block barrier
    // exactly n_my + 1 times, in the same steps.
    if (gatherer) {
        if constexpr (kRmw)
            if (n_my > 0) rmw_prologue(rmw, wave_rows(0), wave_rows(1), wave_rows(2), rpipe);
        if constexpr (kOneHot && !kRmw) onehot_stage_init(stage[w]);
        if constexpr (kOneHot && !kRmw)
            if (n_my > 0)
                onehot_prologue<CO, RPW, true, kBf, NR>(
                    OneHotTiles{wave_rows(0), wave_rows(1), wave_rows(2), -1}, n_in, col_ptr,
                    row_idx, g, dY, pipe);
        if (n_my > 0) load_tile(0, 0);
        __syncthreads();
#pragma unroll 1
        for (int32_t s = 0; s < n_my; ++s) {
            if (s + 1 < n_my) load_tile(s + 1, (s & 1) ^ 1);
            __syncthreads();
        }
        return;
    }

    floatx4 accw[NIB][NWB];
#pragma unroll
    for (int a = 0; a < NIB; ++a)
#pragma unroll
        for (int b = 0; b < NWB; ++b) accw[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};
    // the wave's slice of Wt for dF, held in registers for the whole kernel
    // (it is the same for every tile)
    constexpr bool kWreg = kWLoc == kWRegs;
    static_assert(!kWreg || (kBf ? K2 * WCB <= 512 : K2 * WCB <= 256), "Wt slice too large");
    constexpr int KS = kBf ? K2 / 32 : K2 / 4;  // MFMA k-steps of the dF product
    using BT = typename std::conditional<kBf, bf16x8, float>::type;
    BT bw[kWreg ? KS : 1][WCB];
    if constexpr (kWreg) {
        const int lr = lane >> 4, lc = lane & 15;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int t = 0; t < WCB; ++t) {
                if constexpr (kBf)
                    bw[ks][t] = *reinterpret_cast<const bf16x8 *>(
                        static_cast<const uint16_t *>(Wop) +
                        bt_offset<K2, CI, CO>(16 * (wc + NCBW * t) + lc, 32 * ks + 8 * lr));
                else
                    bw[ks][t] = static_cast<const float *>(
                        Wop)[bt_offset<K2, CI, CO>(16 * (wc + NCBW * t) + lc, 4 * ks + lr)];
            }
    }
    // F rows of tile s (row-major, zero past the last row, 16 B per load) for
    // the dW product, into Fs[s & 1]: the matrix waves load those of the next
    // tile before their products and store them after, so the loads' latency
    // hides behind the products (the gather waves have none of it)
    constexpr int CPR = CI * (int)sizeof(DT) / 16;
    constexpr int NQ = (TR * CPR + kWsMma * 64 - 1) / (kWsMma * 64);
    const int mt = threadIdx.x - kWsGather * 64;  // thread within the matrix role
    auto load_f = [&](int32_t s, uint4 (&val)[NQ]) {
        const int32_t row0 = (t_first + s * gx) * TR;
#pragma unroll
        for (int k = 0; k < NQ; ++k) {
            const int q = mt + k * kWsMma * 64;
            const int r = q / CPR, c16 = q % CPR;
            val[k] = uint4{0u, 0u, 0u, 0u};
            if (q < TR * CPR && row0 + r < n_in)
                val[k] = *reinterpret_cast<const uint4 *>(
                    static_cast<const char *>(Fv) + (int64_t)(row0 + r) * CI * sizeof(DT) +
                    16 * c16);
        }
    };
    auto store_f = [&](int buf, const uint4 (&val)[NQ]) {
#pragma unroll
        for (int k = 0; k < NQ; ++k) {
            const int q = mt + k * kWsMma * 64;
            const int r = q / CPR, c16 = q % CPR;
            if (q < TR * CPR)
                *reinterpret_cast<uint4 *>(reinterpret_cast<char *>(&Fs[buf][r * SF]) +
                                           16 * c16) = val[k];
        }
    };
    if (dW_part && n_my > 0) {
        uint4 val[NQ];
        load_f(0, val);
        store_f(0, val);
    }
    __syncthreads();
#pragma unroll 1
    for (int32_t s = 0; s < n_my; ++s) {
        const int buf = s & 1;
        uint4 fnext[NQ];
        const bool more = dW_part && s + 1 < n_my;
        if (more) load_f(s + 1, fnext);
        {
            const int32_t row0 = (t_first + s * gx) * TR;
            const DT *D = Ds[buf];
            // ---- dF_tile = D_tile Wt  ([TR, K2] x [K2, CI])
            if (dF && mw < NCBW * NRG) {
                floatx4 acc[WRB][WCB];
#pragma unroll
                for (int u = 0; u < WRB; ++u)
#pragma unroll
                    for (int t = 0; t < WCB; ++t) acc[u][t] = floatx4{0.f, 0.f, 0.f, 0.f};
                if constexpr (kWreg) {
                    const int lr = lane >> 4, lc = lane & 15;
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
                        for (int u = 0; u < WRB; ++u) {
                            const int arow = 16 * (wr + NRG * u) + lc;
                            if constexpr (kBf) {
                                const bf16x8 a = *reinterpret_cast<const bf16x8 *>(
                                    &D[arow * SD + 32 * ks + 8 * lr]);
#pragma unroll
                                for (int t = 0; t < WCB; ++t)
                                    acc[u][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                        a, bw[ks][t], acc[u][t], 0, 0, 0);
                            } else {
                                const float a = D[arow * SD + 4 * ks + lr];
#pragma unroll
                                for (int t = 0; t < WCB; ++t)
                                    acc[u][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                                        a, bw[ks][t], acc[u][t], 0, 0, 0);
                            }
                        }
                    }
                } else if constexpr (!kBf) {
                    mfma_lds_x_global_f32t<K2, SD, WRB, WCB, NCBW, NRG, CI, CO>(
                        D, static_cast<const float *>(Wop), wr, wc, acc);
                } else {
                    mfma_lds_x_global_bf16<K2, SD, WRB, WCB, NCBW, NRG, CI, CO>(
                        D, static_cast<const uint16_t *>(Wop), wr, wc, acc);
                }
#pragma unroll
                for (int u = 0; u < WRB; ++u)
#pragma unroll
                    for (int t = 0; t < WCB; ++t)
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            const int32_t row = row0 + 16 * (wr + NRG * u) + 4 * (lane >> 4) + r;
                            if (row < n_in)
                                dF[(int64_t)row * CI + 16 * (wc + NCBW * t) + (lane & 15)] =
                                    acc[u][t][r];
                        }
            }
            // ---- dW += F_tile^T D_tile  ([CI, TR] x [TR, K2]) over the tile rows
            if (dW_part) {
                const DT *Fb = Fs[buf];
                if constexpr (!kBf) {
                    // k-steps of 4 tile rows: in step k lane group lr takes
                    // row (k & 3) + 16 (k >> 2) + 4 lr, so the four rows of
                    // one read sit 4 row strides apart (16 banks apart for
                    // the padded strides); the operands of step k + 1 are
                    // read from LDS while the products of step k run
                    static_assert(TR % 16 == 0, "row permutation covers 16-row blocks");
                    const float *Fp = Fb + 4 * (lane >> 4) * SF + (lane & 15);
                    const float *Dp = D + 4 * (lane >> 4) * SD + 16 * mw * NWB + (lane & 15);
                    float a[2][NIB], bb[2][NWB];
                    auto load_step = [&](int r0, float(&aa)[NIB], float(&bq)[NWB]) {
#pragma unroll
                        for (int ib = 0; ib < NIB; ++ib) aa[ib] = Fp[r0 * SF + 16 * ib];
#pragma unroll
                        for (int nb = 0; nb < NWB; ++nb) bq[nb] = Dp[r0 * SD + 16 * nb];
                    };
                    auto row0_of = [](int k) { return (k & 3) + 16 * (k >> 2); };
                    load_step(0, a[0], bb[0]);
#pragma unroll
                    for (int k = 0; k < TR / 4; ++k) {
                        if (k + 1 < TR / 4) load_step(row0_of(k + 1), a[(k + 1) & 1], bb[(k + 1) & 1]);
                        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                        for (int nb = 0; nb < NWB; ++nb)
#pragma unroll
                            for (int ib = 0; ib < NIB; ++ib)
                                accw[ib][nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                                    a[k & 1][ib], bb[k & 1][nb], accw[ib][nb], 0, 0, 0);
                        __builtin_amdgcn_sched_barrier(0);
                    }
                } else {
#pragma unroll
                    for (int k0 = 0; k0 < TR; k0 += 32) {
                        const int kk = k0 + 8 * (lane >> 4);
                        bf16x8 a[NIB];
#pragma unroll
                        for (int ib = 0; ib < NIB; ++ib)
                            a[ib] = lds_column8(&Fb[kk * SF + 16 * ib + (lane & 15)], SF);
#pragma unroll
                        for (int nb = 0; nb < NWB; ++nb) {
                            const bf16x8 bb =
                                lds_column8(&D[kk * SD + 16 * (mw * NWB + nb) + (lane & 15)], SD);
#pragma unroll
                            for (int ib = 0; ib < NIB; ++ib)
                                accw[ib][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                    a[ib], bb, accw[ib][nb], 0, 0, 0);
                        }
                    }
                }
            }
        }
        if (more) store_f((s + 1) & 1, fnext);
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
                out[(16 * ib + 4 * (lane >> 4) + r) * K2 + 16 * (mw * NWB + nb) + (lane & 15)] =
                    accw[ib][nb][r];
}

// dW[m, c, p] = sum_b part[b, c, m*CO + p].  A block of 256 threads owns
// kReducePos consecutive partial positions, four per thread (16-byte loads);
// its kReduceGroups thread groups each sum a fixed, contiguous range of
// blocks in order (eight loads in flight per thread), and the group sums are
// then added in group order, so the result is independent of scheduling.
constexpr int kReduceGroups = 16;
constexpr int kReducePos = 64;  // 16 threads x 4 positions per group

__global__ void __launch_bounds__(256)
    dw_reduce_kernel(const float *__restrict__ part, int32_t n_parts, int32_t M, int32_t CI,
                     int32_t CO, float *__restrict__ dW) {
    __shared__ float4 sums[kReduceGroups][kReducePos / 4];
    const int64_t K2 = (int64_t)M * CO;
    const int64_t total = (int64_t)CI * K2;  // a multiple of 4 (CO % 16 == 0)
    const int g = threadIdx.x / (kReducePos / 4);
    const int tq = threadIdx.x % (kReducePos / 4);
    const int64_t off = (int64_t)blockIdx.x * kReducePos + 4 * tq;
    const int32_t per = (n_parts + kReduceGroups - 1) / kReduceGroups;
    const int32_t b0 = g * per;
    const int32_t b1 = b0 + per < n_parts ? b0 + per : n_parts;
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    if (off < total) {
        for (int32_t bb = b0; bb < b1; bb += 8) {
            float4 v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j)
                v[j] = bb + j < b1 ? *reinterpret_cast<const float4 *>(
                                         part + (int64_t)(bb + j) * total + off)
                                   : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                s.x += v[j].x;
                s.y += v[j].y;
                s.z += v[j].z;
                s.w += v[j].w;
            }
        }
    }
    sums[g][tq] = s;
    __syncthreads();
    if (g == 0 && off < total) {
        float4 t = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int q = 0; q < kReduceGroups; ++q) {
            const float4 u = sums[q][tq];
            t.x += u.x;
            t.y += u.y;
            t.z += u.z;
            t.w += u.w;
        }
        // off = c*K2 + m*CO + p  ->  dW[(m*CI + c)*CO + p]; p..p+3 share m
        const int64_t c = off / K2, mp = off % K2;
        const int64_t m = mp / CO, p = mp % CO;
        *reinterpret_cast<float4 *>(dW + (m * CI + c) * CO + p) = t;
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
using FwdFn = void (*)(int32_t, const int32_t *, const int32_t *, const float *, KGeo,
                       const void *, const void *, float *);
using RegFn = void (*)(int32_t, int32_t, const int32_t *, const int32_t *, const float *,
                       KGeo, const void *, const void *, float *, const int32_t *);
using BwdFn = void (*)(int32_t, int32_t, const int32_t *, const int32_t *, const int32_t *,
                       const float *, KGeo, const void *, const void *, const void *,
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
        case SBC_BASIS_EVENT_DECAYS + 1:
            if constexpr (M >= 16 && M % 8 == 0)
                return fwd_fused_kernel<M, CI, CO, SBC_BASIS_EVENT_DECAYS + 1, kBf>;
            return nullptr;
    }
    return nullptr;
}

template <int M, int CI, int CO, bool kBf>
RegFn reg_for(int basis_mode) {
    if constexpr (!reg_forward_fits<M, CI, CO, kBf>()) {
        return nullptr;
    } else {
        switch (basis_mode) {
            case 0: return fwd_reg_kernel<M, CI, CO, 0, kBf>;
            case SBC_BASIS_MONO4 + 1:
                if constexpr (M == 4) return fwd_reg_kernel<M, CI, CO, SBC_BASIS_MONO4 + 1, kBf>;
                return nullptr;
            case SBC_BASIS_MONO8 + 1:
                if constexpr (M == 8) return fwd_reg_kernel<M, CI, CO, SBC_BASIS_MONO8 + 1, kBf>;
                return nullptr;
            case SBC_BASIS_EVENT8 + 1:
                if constexpr (M == 8) return fwd_reg_kernel<M, CI, CO, SBC_BASIS_EVENT8 + 1, kBf>;
                return nullptr;
            case SBC_BASIS_EVENT_DECAYS + 1:
                if constexpr (M >= 16 && M % 8 == 0)
                    return fwd_reg_kernel<M, CI, CO, SBC_BASIS_EVENT_DECAYS + 1, kBf>;
                return nullptr;
        }
        return nullptr;
    }
}

template <int M, int CI, int CO, bool kBf>
BwdFn bwd_for(int basis_mode) {
    switch (basis_mode) {
        case 0: return bwd_ws_kernel<M, CI, CO, 0, kBf>;
        case SBC_BASIS_MONO4 + 1:
            if constexpr (M == 4) return bwd_ws_kernel<M, CI, CO, SBC_BASIS_MONO4 + 1, kBf>;
            return nullptr;
        case SBC_BASIS_MONO8 + 1:
            if constexpr (M == 8) return bwd_ws_kernel<M, CI, CO, SBC_BASIS_MONO8 + 1, kBf>;
            return nullptr;
        case SBC_BASIS_EVENT8 + 1:
            if constexpr (M == 8 && CI == 32 && CO == 32 && !kBf)
                return bwd_ws_kernel<M, CI, CO, SBC_BASIS_EVENT8 + 1, kBf, 8, 4, kEventRmwTR,
                                     kWRegs>;
            else if constexpr (M == 8)
                return bwd_ws_kernel<M, CI, CO, SBC_BASIS_EVENT8 + 1, kBf>;
            return nullptr;
        case SBC_BASIS_EVENT_DECAYS + 1:
            if constexpr (M >= 16 && M % 8 == 0)
                return bwd_ws_kernel<M, CI, CO, SBC_BASIS_EVENT_DECAYS + 1, kBf>;
            return nullptr;
        case kDecayDerivMode:
            if constexpr (M >= 16 && M % 8 == 0)
                return bwd_ws_kernel<M, CI, CO, kDecayDerivMode, kBf>;
            return nullptr;
        case kEvent8WideMode:
            if constexpr (M == 8) return bwd_ws_kernel<M, CI, CO, kEvent8WideMode, kBf>;
            return nullptr;
        case kDecaysWideMode:
        case kDecayDerivWideMode:
            // the learned-decay bases through the generic gather (64-bit addressing)
            if constexpr (M >= 16 && M % 8 == 0) {
                constexpr WsCfg c = ws_cfg<M, CI, CO, kBf>();
                if (basis_mode == kDecaysWideMode)
                    return bwd_ws_kernel<M, CI, CO, SBC_BASIS_EVENT_DECAYS + 1, kBf, c.ng, c.nm,
                                         c.tr, c.wloc, false>;
                return bwd_ws_kernel<M, CI, CO, kDecayDerivMode, kBf, c.ng, c.nm, c.tr, c.wloc,
                                     false>;
            }
            return nullptr;
    }
    return nullptr;
}

// Shapes with fused kernels: (M, C_in, C_out, bf16).  The backward keeps a
// C_in x M*C_out partial of dW per block in registers, so its list is limited
// to C_in * M * C_out <= 32768.
#define SBC_FWD_SHAPES(X) \
    X(16, 32, 32, false)  \
    X(10, 64, 64, false)  \
    X(4, 64, 64, false)   \
    X(4, 16, 32, false)   \
    X(8, 64, 64, false)   \
    X(8, 64, 128, false)  \
    X(8, 32, 32, false)   \
    X(8, 64, 64, true)    \
    X(8, 32, 32, true)
#define SBC_BWD_SHAPES(X) \
    X(16, 32, 32, false)  \
    X(4, 64, 64, false)   \
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

RegFn find_reg(const Shape &s, int basis_mode) {
#define SBC_X(m_, ci_, co_, bf_) \
    if (s.M == m_ && s.CI == ci_ && s.CO == co_ && s.bf == bf_) return reg_for<m_, ci_, co_, bf_>(basis_mode);
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

// ws_cfg() of a shape listed for the fused kernels
WsCfg ws_cfg_rt(int32_t M, int32_t CI, int32_t CO, bool bf) {
#define SBC_X(m_, ci_, co_, bf_) \
    if (M == m_ && CI == ci_ && CO == co_ && bf == bf_) return ws_cfg<m_, ci_, co_, bf_>();
    SBC_BWD_SHAPES(SBC_X)
#undef SBC_X
    return WsCfg{4, 4, 32, kWGlobal};
}

int basis_mode_of(const float *v, const sbc_geometry *g) {
    return v ? 0 : (int)g->basis + 1;
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

// Workspace of the fused kernels: a permuted copy of W, the per-block dW
// partials, the packed event coordinates, and for M = 10 (the weighted basis,
// whose values need whole rows) the materialised basis values.
size_t fused_workspace_bytes(int32_t M, int32_t CI, int32_t CO, int32_t n_points, int64_t nnz) {
    return align_up((size_t)M * CI * CO * 4) +
           align_up((size_t)kMaxBlocksBwd * (size_t)CI * M * CO * 4) +
           align_up((size_t)(n_points > 0 ? n_points : 0) * sizeof(int4)) +
           (M == 10 ? align_up((size_t)(nnz > 0 ? nnz : 0) * M * 4) : 0);
}

// The forward needs no dW partials: the weight copy, the packed events, the
// row order of the register-resident forward and (M = 10) the basis values.
size_t fused_forward_workspace_bytes(int32_t M, int32_t CI, int32_t CO, int32_t n_points,
                                     int64_t nnz) {
    const size_t n = (size_t)(n_points > 0 ? n_points : 0);
    return align_up((size_t)M * CI * CO * 4) + align_up(n * sizeof(int4)) +
           align_up(n * sizeof(int32_t)) +
           (M == 10 ? align_up((size_t)(nnz > 0 ? nnz : 0) * M * 4) : 0);
}

namespace {

// Kernel geometry for a call: packs the event coordinates into the workspace
// (after the weight copy and the dW partials) when the basis is evaluated
// from an event stream.
// ev_offset: where the packed events go in the workspace.
sbc_status make_kgeo(const sbc_csr *csr, const float *v, const sbc_geometry *g, size_t ev_offset,
                     void *ws, hipStream_t stream, KGeo *kg) {
    *kg = KGeo{};
    kg->nnz = csr->nnz_bound > INT32_MAX ? INT32_MAX : (int32_t)csr->nnz_bound;
    if (v || !g) return SBC_OK;
    kg->inv_r = 1.0 / (double)g->radius;
    kg->inv_tau = 1.0f / g->tau;
    kg->x_in = g->x_in;
    kg->x_out = g->x_out;
    kg->decays = g->decays;
    if (g->basis == SBC_BASIS_EVENT8 || g->basis == SBC_BASIS_EVENT_DECAYS) {
        // event streams are in place: rows and columns index the same events
        const int32_t n = csr->n_cols > csr->n_rows ? csr->n_cols : csr->n_rows;
        int4 *pk = reinterpret_cast<int4 *>(static_cast<char *>(ws) + ev_offset);
        if (n > 0) {
            int blocks = grid_for(n, 256);
            if (blocks > 2048) blocks = 2048;
            hipLaunchKernelGGL(pack_events_kernel, dim3(blocks), dim3(256), 0, stream, g->px, g->py,
                               g->t, n, pk);
            SBC_LAUNCH_CHECK();
        }
        kg->ev = pk;
    }
    return SBC_OK;
}

}  // namespace

sbc_status fused_forward(const sbc_csr *csr, const float *v, const sbc_geometry *g, int32_t M,
                         const void *F, const void *W, bool bf, int32_t CI, int32_t CO, float *Y,
                         void *ws, hipStream_t stream) {
    if (!v && g->basis == SBC_BASIS_WMONO10) {
        // row-normalised values: materialised first, behind the other regions
        const int32_t n = csr->n_cols > csr->n_rows ? csr->n_cols : csr->n_rows;
        float *vm = reinterpret_cast<float *>(
            static_cast<char *>(ws) + fused_forward_workspace_bytes(M, CI, CO, n, 0));
        SBC_TRY(basis_eval_launch(csr, g, vm, stream));
        v = vm;
    }
    FwdFn fn = find_fwd(Shape{M, CI, CO, bf}, basis_mode_of(v, g));
    if (!fn) return fail(SBC_ERR_UNSUPPORTED, "no fused forward for this shape");
    if (csr->n_rows == 0) return SBC_OK;
    KGeo gr;
    // layout: [W copy][packed events][row order][M = 10: basis values]
    SBC_TRY(make_kgeo(csr, v, g, align_up((size_t)M * CI * CO * 4), ws, stream, &gr));
    RegFn rf = find_reg(Shape{M, CI, CO, bf}, basis_mode_of(v, g));
    // the fixed-decay event basis on rows of 32 float32 channels: the one-hot
    // forward, whose loads take 32-bit byte offsets (F rows, packed events and
    // the pattern's indices under 4 GiB; else, or with SBC_EVENT8_WIDE_PATH=1,
    // the register forward)
    bool onehot = basis_mode_of(v, g) == SBC_BASIS_EVENT8 + 1 && M == 8 && CI == 32 &&
                  CO == 32 && !bf;
    if (onehot) {
        const int64_t n_ev = csr->n_cols > csr->n_rows ? csr->n_cols : csr->n_rows;
        const int64_t lim = (int64_t)1 << 32;
        const char *force = std::getenv("SBC_EVENT8_WIDE_PATH");
        if ((int64_t)csr->n_cols * CI * 4 >= lim || n_ev * 16 >= lim ||
            csr->nnz_bound * 4 >= lim || csr->nnz_bound < 1 || (force && force[0] == '1'))
            onehot = false;
    }
    if (rf || onehot) {
        const int32_t n_tiles = (csr->n_rows + 15) / 16;
        const int32_t np = csr->n_cols > csr->n_rows ? csr->n_cols : csr->n_rows;
        int32_t *order = reinterpret_cast<int32_t *>(
            static_cast<char *>(ws) + align_up((size_t)M * CI * CO * 4) +
            align_up((size_t)np * sizeof(int4)));
        hipLaunchKernelGGL(row_order_kernel,
                           dim3(grid_for(csr->n_rows, kOrderWindow * (kOrderThreads / 64))),
                           dim3(kOrderThreads), 0, stream, csr->n_rows, csr->row_ptr, gr.nnz,
                           order);
        SBC_LAUNCH_CHECK();
        if (onehot) {
            // one block per CU (its LDS holds W and the eight waves' G slots)
            int blocks = (n_tiles + kOhWaves - 1) / kOhWaves;
            if (blocks > device_cus()) blocks = device_cus();
            trace_before("fwd_fused", stream);
            hipLaunchKernelGGL((fwd_onehot_kernel<32, 32>), dim3(blocks), dim3(kOhWaves * 64), 0,
                               stream, csr->n_rows, n_tiles, csr->row_ptr, csr->col_idx, gr,
                               static_cast<const float *>(F), static_cast<const float *>(W), Y,
                               order);
            SBC_LAUNCH_CHECK();
            trace_after("fwd_fused", stream);
            return SBC_OK;
        }
        int per_cu = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void *>(rf),
                                                         kRegWaves * 64, 0) != hipSuccess ||
            per_cu < 1)
            per_cu = 1;
        int blocks = (n_tiles + kRegWaves - 1) / kRegWaves;
        if (blocks > device_cus() * per_cu) blocks = device_cus() * per_cu;
        trace_before("fwd_fused", stream);
        hipLaunchKernelGGL(rf, dim3(blocks), dim3(kRegWaves * 64), 0, stream, csr->n_rows,
                           n_tiles, csr->row_ptr, csr->col_idx, v, gr, F, W, Y, order);
        SBC_LAUNCH_CHECK();
        trace_after("fwd_fused", stream);
        return SBC_OK;
    }
    // W transposed, [CO, K]: element (m, c, p) at p*K + m*CI + c (float32 or bf16)
    SBC_TRY(launch_perm(W, bf, bf, M, CI, CO, CI, 1, (int64_t)M * CI, ws, stream));
    const void *Wop = ws;
    const int K = M * CI;
    const int TR = fwd_tile_rows(K, CO, bf);
    trace_before("fwd_fused", stream);
    hipLaunchKernelGGL(fn, dim3(grid_for(csr->n_rows, TR)), dim3(kFwdWaves * 64), 0, stream,
                       csr->n_rows, csr->row_ptr, csr->col_idx, v, gr, F, Wop, Y);
    SBC_LAUNCH_CHECK();
    trace_after("fwd_fused", stream);
    return SBC_OK;
}

sbc_status fused_backward(const sbc_csr *csr, const sbc_csc *csc, const float *v,
                          const sbc_geometry *g, int32_t M, const void *F, const void *W,
                          const void *dY, bool bf, int32_t CI, int32_t CO, float *dF, float *dW,
                          void *ws, hipStream_t stream, bool decay_derivative) {
    int mode = decay_derivative ? kDecayDerivMode : basis_mode_of(v, g);
    if (mode == SBC_BASIS_EVENT8 + 1) {
        // the one-hot gather's 32-bit byte offsets: dY rows, packed events,
        // the pattern's indices and column bounds under 4 GiB.  The
        // environment variable SBC_EVENT8_WIDE_PATH=1 takes the other path at
        // any size (so that tests can run it).
        const int64_t n_ev = csr->n_cols > csr->n_rows ? csr->n_cols : csr->n_rows;
        const int64_t lim = (int64_t)1 << 32;
        const char *force = std::getenv("SBC_EVENT8_WIDE_PATH");
        if ((int64_t)csr->n_rows * CO * (bf ? 2 : 4) >= lim || n_ev * 16 >= lim ||
            csr->nnz_bound * 4 >= lim || ((int64_t)csr->n_cols + 1) * 4 >= lim ||
            csr->nnz_bound < 1 || (force && force[0] == '1'))
            mode = kEvent8WideMode;
    }
    if (mode == SBC_BASIS_EVENT_DECAYS + 1 || mode == kDecayDerivMode) {
        // the learned decays' in-place gather: the same limits
        const int64_t n_ev = csr->n_cols > csr->n_rows ? csr->n_cols : csr->n_rows;
        const int64_t lim = (int64_t)1 << 32;
        const char *force = std::getenv("SBC_EVENT8_WIDE_PATH");
        if ((int64_t)csr->n_rows * CO * (bf ? 2 : 4) >= lim || n_ev * 16 >= lim ||
            csr->nnz_bound * 4 >= lim || ((int64_t)csr->n_cols + 1) * 4 >= lim ||
            csr->nnz_bound < 1 || (force && force[0] == '1'))
            mode = mode == kDecayDerivMode ? kDecayDerivWideMode : kDecaysWideMode;
    }
    BwdFn fn = find_bwd(Shape{M, CI, CO, bf}, mode);
    if (!fn) return fail(SBC_ERR_UNSUPPORTED, "no fused backward for this shape");
    const int32_t n_in = csr->n_cols;
    char *base = static_cast<char *>(ws);
    float *part = reinterpret_cast<float *>(base + align_up((size_t)M * CI * CO * 4));
    // the kernel reads W [M, CI, CO] in place as Wt [CI, M*CO]
    const WsCfg cfg = ws_cfg_rt(M, CI, CO, bf);
    const int TR = mode == SBC_BASIS_EVENT8 + 1 && M == 8 && CI == 32 && CO == 32 && !bf
                       ? kEventRmwTR
                       : cfg.tr;
    const int32_t n_tiles = (n_in + TR - 1) / TR;
    const int nw = cfg.ng + cfg.nm;
    int blocks = device_cus();
    if (blocks > kMaxBlocksBwd) blocks = kMaxBlocksBwd;
    if (blocks > n_tiles) blocks = n_tiles;
    if (blocks < 1) blocks = 1;
    KGeo gg;
    // layout: [W copy][dW partials][packed events]
    SBC_TRY(make_kgeo(csr, v, g,
                      align_up((size_t)M * CI * CO * 4) +
                          align_up((size_t)kMaxBlocksBwd * (size_t)CI * M * CO * 4),
                      ws, stream, &gg));
    if (n_in > 0 && (dF || dW)) {
        trace_before(decay_derivative ? "decay_fused" : "bwd_fused", stream);
        hipLaunchKernelGGL(fn, dim3(blocks), dim3(nw * 64), 0, stream, n_in, n_tiles, csc->col_ptr,
                           csc->row_idx, csc->edge_perm, v, gg, F, dY, W, dF,
                           dW ? part : nullptr);
        SBC_LAUNCH_CHECK();
        trace_after(decay_derivative ? "decay_fused" : "bwd_fused", stream);
    }
    if (!dW) return SBC_OK;
    const int64_t total = (int64_t)M * CI * CO;
    const int64_t rb = (total + kReducePos - 1) / kReducePos;
    trace_before(decay_derivative ? "decay_dw_reduce" : "bwd_dw_reduce", stream);
    hipLaunchKernelGGL(dw_reduce_kernel, dim3((unsigned)rb), dim3(256), 0, stream, part,
                       n_in > 0 ? blocks : 0, M, CI, CO, dW);
    SBC_LAUNCH_CHECK();
    trace_after(decay_derivative ? "decay_dw_reduce" : "bwd_dw_reduce", stream);
    return SBC_OK;
}

}  // namespace sbc
