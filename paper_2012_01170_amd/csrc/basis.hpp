// Basis functions p_m of the neighbourhood matrices, evaluated per edge on the
// device (Section 3.1: the entries of N^(m) are the basis functions at the
// edge vector; the paper computes them on the accelerator from the neighbour
// indices).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "../../include/sbconv.h"

namespace sbc {

// Point monomials of u = (x'_i - x_j) / r times the window (1 - |u|^2)^2.
// M = 4: [1, ux, uy, uz];  M = 8: [1, ux, uy, uz, ux^2, uy^2, uz^2, ux*uy].
// Evaluated in float64 and rounded once: the coordinate differences are then
// exact and 1 - |u|^2 keeps its relative accuracy near the ball's edge, where
// float32 would cancel.
template <int M>
__device__ __forceinline__ void point_basis(float qx, float qy, float qz, float px, float py,
                                            float pz, double inv_r, float *v) {
    const double ux = ((double)qx - (double)px) * inv_r;
    const double uy = ((double)qy - (double)py) * inv_r;
    const double uz = ((double)qz - (double)pz) * inv_r;
    const double a = 1.0 - (ux * ux + uy * uy + uz * uz);
    const double w = a * a;
    v[0] = (float)w;
    v[1] = (float)(ux * w);
    v[2] = (float)(uy * w);
    v[3] = (float)(uz * w);
    if constexpr (M == 8) {
        v[4] = (float)(ux * ux * w);
        v[5] = (float)(uy * uy * w);
        v[6] = (float)(uz * uz * w);
        v[7] = (float)(ux * uy * w);
    }
}

// Weighted convolution (Section 3.1, Eq. 11) with every monomial up to second
// order: an edge's weight w = 1 - |dx| / r, which falls to zero at the ball
// radius, and its ten monomials of u = dx / r times s (= w / W_i, the row's
// normaliser), as float32: [1, ux, uy, uz, ux^2, uy^2, uz^2, ux*uy, ux*uz,
// uy*uz].  Differences are taken in float64 from the float32 coordinates.
__device__ __forceinline__ double point_weight(float qx, float qy, float qz, float px, float py,
                                               float pz, double inv_r) {
    const double dx = (double)qx - (double)px, dy = (double)qy - (double)py,
                 dz = (double)qz - (double)pz;
    return 1.0 - sqrt(dx * dx + dy * dy + dz * dz) * inv_r;
}

__device__ __forceinline__ void weighted_mono10(float qx, float qy, float qz, float px, float py,
                                                float pz, double inv_r, double s, float *v) {
    const double ux = ((double)qx - (double)px) * inv_r;
    const double uy = ((double)qy - (double)py) * inv_r;
    const double uz = ((double)qz - (double)pz) * inv_r;
    v[0] = (float)s;
    v[1] = (float)(ux * s);
    v[2] = (float)(uy * s);
    v[3] = (float)(uz * s);
    v[4] = (float)(ux * ux * s);
    v[5] = (float)(uy * uy * s);
    v[6] = (float)(uz * uz * s);
    v[7] = (float)(ux * uy * s);
    v[8] = (float)(ux * uz * s);
    v[9] = (float)(uy * uz * s);
}

// Basis size of a geometry (8 n_decays for the learned-decay event kernel).
inline int32_t geometry_basis_size(const sbc_geometry &g) {
    if (g.basis == SBC_BASIS_EVENT_DECAYS) return 8 * g.n_decays;
    switch (g.basis) {
        case SBC_BASIS_MONO4: return 4;
        case SBC_BASIS_MONO8:
        case SBC_BASIS_EVENT8: return 8;
        case SBC_BASIS_WMONO10: return 10;
        default: return 0;
    }
}

// Event basis: index of pixel offset u = (ux, uy) in the 3x3 block, row-major
// over (uy, ux) with the centre removed; -1 for the centre (and for offsets
// outside the block, which no neighbourhood produces).
__device__ __forceinline__ int event_index(int32_t ux, int32_t uy) {
    // (without branches: ux + 1 and uy + 1 are in 0..2 exactly when their
    // unsigned forms are at most 2)
    const uint32_t bx = (uint32_t)ux + 1u, by = (uint32_t)uy + 1u;
    const int k = (int)(by * 3u + bx);
    return (bx <= 2u && by <= 2u && k != 4) ? k - (k > 4 ? 1 : 0) : -1;
}

// exp(-dt / tau) for an integer time gap dt >= 0.  The gap is converted to
// float from its int32 difference when that does not overflow (the same
// value, rounded once), else from the int64 one.
__device__ __forceinline__ float event_decay(int32_t ti, int32_t tj, float inv_tau) {
    const int32_t d = (int32_t)((uint32_t)ti - (uint32_t)tj);
    float dt;
    if (__builtin_expect(((ti ^ tj) & (ti ^ d)) < 0, 0))
        dt = (float)((int64_t)ti - (int64_t)tj);
    else
        dt = (float)d;
    return expf(-dt * inv_tau);
}

}  // namespace sbc
