// sbc_conv_forward / sbc_conv_backward: Y = sum_m N^(m) F W^(m) and its
// gradients (Section 3.1, the matrix-product form; its down- and up-sampling
// evaluation orders and their multiply-add counts).
//
// Forward, SpMM-first ((N F) W):  G = [N^(m) F]_m [n_out, M*C_in] (gather), Y = G W_flat (MFMA)
// Forward, GEMM-first (N (F W)):  H = F [W^(m)]_m [n_in, M*C_out] (MFMA), Y = sum_m N^(m) H_m
// Backward, D-route (gather first):  D = [N^(m)T dY]_m [n_in, M*C_out], dF = D Wt, dW = F^T D
// Backward, G-route (GEMM first):    dG = dY W_flat^T, dF = N^T dG; dW = G^T dY with G = N F
// Shapes listed in fused.hip run SpMM-first forward and the D-route as fused
// kernels (basis evaluated inside); other shapes and orders use the generic
// kernels below, which evaluate the basis into the workspace first when v is
// NULL.
#include <mutex>
#include <string>

#include "basis.hpp"
#include "common.hpp"
#include "fused.hpp"
#include "gemm.hpp"
#include "spmm.hpp"

namespace sbc {
namespace {

__device__ __forceinline__ float ldw(const float *p, int64_t i) { return p[i]; }
__device__ __forceinline__ float ldw(const uint16_t *p, int64_t i) {
    return __uint_as_float((uint32_t)p[i] << 16);
}

// W [M, Ci, Co] -> out with element (m, c, p) at m*s_m + c*s_c + p*s_p, as float32.
template <typename T>
__global__ void permute_w_kernel(const T *__restrict__ W, int32_t M, int32_t Ci, int32_t Co,
                                 int64_t s_m, int64_t s_c, int64_t s_p, float *__restrict__ out) {
    const int64_t total = (int64_t)M * Ci * Co;
    for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < total;
         x += (int64_t)gridDim.x * blockDim.x) {
        const int32_t p = (int32_t)(x % Co);
        const int32_t c = (int32_t)((x / Co) % Ci);
        const int32_t m = (int32_t)(x / ((int64_t)Co * Ci));
        out[m * s_m + c * s_c + p * s_p] = ldw(W, x);
    }
}

sbc_status permute_w(const void *W, bool bf16, int32_t M, int32_t Ci, int32_t Co, int64_t s_m,
                     int64_t s_c, int64_t s_p, float *out, hipStream_t stream) {
    int64_t total = (int64_t)M * Ci * Co;
    int64_t blocks = (total + 255) / 256;
    if (blocks > 1024) blocks = 1024;
    if (bf16)
        hipLaunchKernelGGL(permute_w_kernel<uint16_t>, dim3((unsigned)blocks), dim3(256), 0, stream,
                           static_cast<const uint16_t *>(W), M, Ci, Co, s_m, s_c, s_p, out);
    else
        hipLaunchKernelGGL(permute_w_kernel<float>, dim3((unsigned)blocks), dim3(256), 0, stream,
                           static_cast<const float *>(W), M, Ci, Co, s_m, s_c, s_p, out);
    SBC_LAUNCH_CHECK();
    return SBC_OK;
}

// dwp [C_in, M, C_out] -> dW [M, C_in, C_out]
__global__ void permute_back_kernel(const float *__restrict__ dwp, int32_t M, int32_t Ci,
                                    int32_t Co, float *__restrict__ dW) {
    const int64_t total = (int64_t)M * Ci * Co;
    for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < total;
         x += (int64_t)gridDim.x * blockDim.x) {
        const int32_t p = (int32_t)(x % Co);
        const int32_t c = (int32_t)((x / Co) % Ci);
        const int32_t m = (int32_t)(x / ((int64_t)Co * Ci));
        dW[x] = dwp[((int64_t)c * M + m) * Co + p];
    }
}

sbc_status permute_w_back(const float *dwp, int32_t M, int32_t Ci, int32_t Co, float *dW,
                          hipStream_t stream) {
    int64_t total = (int64_t)M * Ci * Co;
    int64_t blocks = (total + 255) / 256;
    if (blocks > 1024) blocks = 1024;
    hipLaunchKernelGGL(permute_back_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, dwp, M,
                       Ci, Co, dW);
    SBC_LAUNCH_CHECK();
    return SBC_OK;
}

// Routes of the four products.  Forward: SpMM-first gathers G = N F then
// contracts with W; GEMM-first contracts H = F W then gathers over H.
// Backward: the D-route gathers D = N^T dY first (dF = D Wt, dW = F^T D), the
// G-route contracts dG = dY W^T first (dF = N^T dG) with dW = G^T dY.
enum Route { kFwdSpmm, kFwdGemm, kBwdD, kBwdG };

struct ConvWs {
    float *v;        // [nnz, M] basis values (when not supplied)
    float *inter;    // G / H / D
    float *inter2;   // dG (G-route)
    float *wperm;    // permuted weights
    float *dwperm;   // dW in [C_in, M, C_out] (D-route)
    float *partial;  // split-K partial tiles
};

ConvWs carve_route(void *base, Route r, int32_t n_out, int32_t n_in, int64_t nnz, int32_t M,
                   int32_t Ci, int32_t Co, size_t *bytes) {
    Carver cv(base);
    ConvWs w{};
    w.v = cv.take<float>((size_t)nnz * M);
    const int64_t wsz = (int64_t)M * Ci * Co;
    size_t p = 0;
    auto upd = [&p](size_t q) { p = q > p ? q : p; };
    switch (r) {
        case kFwdSpmm:
            w.inter = cv.take<float>((size_t)n_out * M * Ci);
            upd(gemm_workspace_floats(n_out, Co, (int64_t)M * Ci));
            break;
        case kFwdGemm:
            w.inter = cv.take<float>((size_t)n_in * M * Co);
            w.wperm = cv.take<float>((size_t)wsz);
            upd(gemm_workspace_floats(n_in, M * Co, Ci));
            break;
        case kBwdD:
            w.inter = cv.take<float>((size_t)n_in * M * Co);
            w.wperm = cv.take<float>((size_t)wsz);
            w.dwperm = cv.take<float>((size_t)wsz);
            upd(gemm_workspace_floats(n_in, Ci, (int64_t)M * Co));
            upd(gemm_workspace_floats(Ci, M * Co, n_in));
            break;
        case kBwdG:
            w.inter = cv.take<float>((size_t)n_out * M * Ci);
            w.inter2 = cv.take<float>((size_t)n_out * M * Ci);
            upd(gemm_workspace_floats(M * Ci, Co, n_out));
            upd(gemm_workspace_floats(n_out, M * Ci, Co));
            break;
    }
    w.partial = cv.take<float>(p);
    if (bytes) *bytes = cv.used;
    return w;
}

bool route_fused(Route r, int32_t M, int32_t Ci, int32_t Co, bool bf) {
    if (r == kFwdSpmm) return fused_forward_available(M, Ci, Co, bf);
    if (r == kBwdD) return fused_backward_available(M, Ci, Co, bf);
    return false;
}

size_t route_bytes(Route r, int32_t n_out, int32_t n_in, int64_t nnz, int32_t M, int32_t Ci,
                   int32_t Co, bool bf) {
    if (route_fused(r, M, Ci, Co, bf))
        return r == kFwdSpmm
                   ? fused_forward_workspace_bytes(M, Ci, Co, n_out > n_in ? n_out : n_in, nnz)
                   : fused_workspace_bytes(M, Ci, Co, n_out > n_in ? n_out : n_in, nnz);
    size_t b = 0;
    carve_route(nullptr, r, n_out, n_in, nnz, M, Ci, Co, &b);
    return b;
}

// AUTO: the order with the lower estimated cost, the multiply-adds of the
// paper's cost table plus a fixed cost per kernel launch (kLaunchMacs, about
// 5 us of launch and dependency latency at 1e13 multiply-adds/s, as measured
// with rocprofv3 on MI355X), a fused pass counting as kFusedLaunches and a
// pass of separate gather and contraction kernels as kSplitLaunches.  The
// launch term only decides between orders whose multiply-adds differ by less
// than a few launches' worth, i.e. small problems, where the fused pass wins.
constexpr double kLaunchMacs = 5e7;
constexpr double kFusedLaunches = 2, kSplitLaunches = 5;

double order_macs(int32_t n_out, int32_t n_in, int64_t nnz, int32_t M, int32_t Ci, int32_t Co,
                  bool spmm_first) {
    const double E = (double)(nnz > 0 ? nnz : 0);
    return spmm_first ? (double)M * Ci * (E + (double)n_out * Co)
                      : (double)M * Co * (E + (double)n_in * Ci);
}

Route forward_route(int32_t n_out, int32_t n_in, int64_t nnz, int32_t M, int32_t Ci, int32_t Co,
                    sbc_order order, bool bf) {
    if (order == SBC_ORDER_SPMM_FIRST) return kFwdSpmm;
    if (order == SBC_ORDER_GEMM_FIRST) return kFwdGemm;
    const double spmm = order_macs(n_out, n_in, nnz, M, Ci, Co, true) +
                        kLaunchMacs * (route_fused(kFwdSpmm, M, Ci, Co, bf) ? kFusedLaunches
                                                                             : kSplitLaunches);
    const double gemm = order_macs(n_out, n_in, nnz, M, Ci, Co, false) +
                        kLaunchMacs * kSplitLaunches;
    return spmm <= gemm ? kFwdSpmm : kFwdGemm;
}

// The backward is itself a convolution from the outputs back to the inputs
// (N^T, channels C_out -> C_in); AUTO applies the same estimate to it.
// Explicit orders name what is done first: SPMM_FIRST = D-route, GEMM_FIRST = G-route.
Route backward_route(int32_t n_out, int32_t n_in, int64_t nnz, int32_t M, int32_t Ci, int32_t Co,
                     sbc_order order, bool bf) {
    if (order == SBC_ORDER_SPMM_FIRST) return kBwdD;
    if (order == SBC_ORDER_GEMM_FIRST) return kBwdG;
    const double d = order_macs(n_in, n_out, nnz, M, Co, Ci, true) +
                     kLaunchMacs * (route_fused(kBwdD, M, Ci, Co, bf) ? kFusedLaunches
                                                                       : kSplitLaunches);
    const double g = order_macs(n_in, n_out, nnz, M, Co, Ci, false) +
                     kLaunchMacs * kSplitLaunches;
    return d <= g ? kBwdD : kBwdG;
}

// feature, weight and gradient rows are moved 16 bytes at a time
bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

sbc_status check_conv_args(const sbc_csr *csr, const float *v, const sbc_geometry *g, int32_t M,
                           const void *F, const void *W, sbc_dtype dtype, int32_t Ci, int32_t Co) {
    SBC_TRY(check_csr(csr));
    if (M != 4 && M != 8 && M != 10 && M != 16 && M != 24 && M != 32)
        return fail(SBC_ERR_UNSUPPORTED, "M must be 4, 8, 10, 16, 24 or 32");
    if (Ci <= 0 || Co <= 0) return fail(SBC_ERR_INVALID_ARG, "C_in and C_out must be > 0");
    if (dtype != SBC_F32 && dtype != SBC_BF16) return fail(SBC_ERR_INVALID_ARG, "unknown dtype");
    if (!W || (csr->n_cols > 0 && !F)) return fail(SBC_ERR_INVALID_ARG, "F or W is null");
    if (!aligned16(F) || !aligned16(W))
        return fail(SBC_ERR_INVALID_ARG, "F and W must be 16-byte aligned");
    if (!v) {
        SBC_TRY(check_geometry(g, csr->n_rows, csr->n_cols));
        if (geometry_basis_size(*g) != M)
            return fail(SBC_ERR_INVALID_ARG, "M does not match the geometry's basis");
    }
    return SBC_OK;
}

sbc_status check_order(sbc_order order) {
    if (order != SBC_ORDER_AUTO && order != SBC_ORDER_SPMM_FIRST && order != SBC_ORDER_GEMM_FIRST)
        return fail(SBC_ERR_INVALID_ARG, "unknown order");
    return SBC_OK;
}

}  // namespace
}  // namespace sbc

using namespace sbc;

extern "C" sbc_order sbc_resolve_order(int32_t n_out, int32_t n_in, int64_t nnz, int32_t M,
                                       int32_t C_in, int32_t C_out, sbc_order order) {
    if (order == SBC_ORDER_SPMM_FIRST || order == SBC_ORDER_GEMM_FIRST) return order;
    // multiply-adds of the two orders (the paper's cost table):
    //   (N F) W:  M C_in (E + n_out C_out);   N (F W):  M C_out (E + n_in C_in)
    return order_macs(n_out, n_in, nnz, M, C_in, C_out, true) <=
                   order_macs(n_out, n_in, nnz, M, C_in, C_out, false)
               ? SBC_ORDER_SPMM_FIRST
               : SBC_ORDER_GEMM_FIRST;
}

extern "C" sbc_status sbc_conv_plan(int32_t n_out, int32_t n_in, int64_t nnz_bound, int32_t M,
                                    int32_t C_in, int32_t C_out, sbc_dtype dtype, sbc_order order,
                                    sbc_conv_plan_t *plan) {
    clear_error();
    if (!plan) return fail(SBC_ERR_INVALID_ARG, "plan is null");
    if (n_out < 0 || n_in < 0 || nnz_bound < 0 || M <= 0 || C_in <= 0 || C_out <= 0)
        return fail(SBC_ERR_INVALID_ARG, "negative or zero size");
    SBC_TRY(check_order(order));
    const bool bf = dtype == SBC_BF16;
    const Route f = forward_route(n_out, n_in, nnz_bound, M, C_in, C_out, order, bf);
    const Route b = backward_route(n_out, n_in, nnz_bound, M, C_in, C_out, order, bf);
    plan->forward_order = f == kFwdSpmm ? SBC_ORDER_SPMM_FIRST : SBC_ORDER_GEMM_FIRST;
    plan->backward_order = b == kBwdD ? SBC_ORDER_SPMM_FIRST : SBC_ORDER_GEMM_FIRST;
    plan->forward_fused = route_fused(f, M, C_in, C_out, bf) ? 1 : 0;
    plan->backward_fused = route_fused(b, M, C_in, C_out, bf) ? 1 : 0;
    return SBC_OK;
}

extern "C" size_t sbc_conv_workspace_size(int32_t n_out, int32_t n_in, int64_t nnz_bound,
                                          int32_t M, int32_t C_in, int32_t C_out,
                                          sbc_dtype dtype, sbc_order order) {
    if (n_out < 0 || n_in < 0 || nnz_bound < 0 || M <= 0 || C_in <= 0 || C_out <= 0) return 0;
    const bool bf = dtype == SBC_BF16;
    const Route f = forward_route(n_out, n_in, nnz_bound, M, C_in, C_out, order, bf);
    const Route b = backward_route(n_out, n_in, nnz_bound, M, C_in, C_out, order, bf);
    const size_t a = route_bytes(f, n_out, n_in, nnz_bound, M, C_in, C_out, bf);
    const size_t c = route_bytes(b, n_out, n_in, nnz_bound, M, C_in, C_out, bf);
    return a > c ? a : c;
}

namespace sbc {
namespace {

// The forward pass with its temporary space in `workspace` (workspace_bytes of it).
sbc_status conv_forward(const sbc_csr *csr, const float *v, const sbc_geometry *geometry,
                        int32_t M, const void *F, const void *W, sbc_dtype dtype, int32_t C_in,
                        int32_t C_out, float *Y, sbc_order order, void *workspace,
                        size_t workspace_bytes, hipStream_t stream) {
    SBC_TRY(check_conv_args(csr, v, geometry, M, F, W, dtype, C_in, C_out));
    SBC_TRY(check_order(order));
    if (!Y && csr->n_rows > 0) return fail(SBC_ERR_INVALID_ARG, "Y is null");
    if (!aligned16(Y)) return fail(SBC_ERR_INVALID_ARG, "Y must be 16-byte aligned");
    const int32_t n_out = csr->n_rows, n_in = csr->n_cols;
    const bool bf = dtype == SBC_BF16;
    const Route r = forward_route(n_out, n_in, csr->nnz_bound, M, C_in, C_out, order, bf);
    const size_t need = route_bytes(r, n_out, n_in, csr->nnz_bound, M, C_in, C_out, bf);
    if (!workspace || workspace_bytes < need)
        return fail(SBC_ERR_WORKSPACE, "workspace smaller than sbc_conv_workspace_size()");
    if (route_fused(r, M, C_in, C_out, bf))
        return fused_forward(csr, v, geometry, M, F, W, bf, C_in, C_out, Y, workspace, stream);

    ConvWs ws = carve_route(workspace, r, n_out, n_in, csr->nnz_bound, M, C_in, C_out, nullptr);
    const float *vv = v;
    if (!vv) {
        SBC_TRY(basis_eval_launch(csr, geometry, ws.v, stream));
        vv = ws.v;
    }
    if (r == kFwdSpmm) {
        SBC_TRY(spmm(n_out, csr->row_ptr, csr->col_idx, nullptr, vv, M, F, bf, C_in, false,
                     csr->nnz_bound, ws.inter, stream, "fwd_spmm"));
        SBC_TRY(gemm(ws.inter, false, (int64_t)M * C_in, 1, W, bf, C_out, 1, Y, C_out, 1, n_out,
                     C_out, (int64_t)M * C_in, ws.partial, stream, "fwd_gemm"));
    } else {
        // Wp [C_in, M, C_out]
        SBC_TRY(permute_w(W, bf, M, C_in, C_out, C_out, (int64_t)M * C_out, 1, ws.wperm, stream));
        SBC_TRY(gemm(F, bf, C_in, 1, ws.wperm, false, (int64_t)M * C_out, 1, ws.inter,
                     (int64_t)M * C_out, 1, n_in, M * C_out, C_in, ws.partial, stream,
                     "fwd_gemm_h"));
        SBC_TRY(spmm(n_out, csr->row_ptr, csr->col_idx, nullptr, vv, M, ws.inter, false, C_out,
                     true, csr->nnz_bound, Y, stream, "fwd_spmm_contract"));
    }
    return SBC_OK;
}

// ---------------------------------------------------------------- forward without allocation
// Device memory of this library's own, for callers that cannot allocate: a
// file-scope array that every GPU the library runs on holds for the life of
// the process.  In host code `scratch` only names the symbol; its address on
// the current device comes from hipGetSymbolAddress, taken once per device
// (each device holds its own copy) and kept in g_scratch.
constexpr size_t kScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch[kMaxDevices] = {};

// This device's scratch address (the symbol lookup runs on the first call on
// each device, with that device current).
sbc_status scratch_of_current_device(void **out) {
    int dev = 0;
    SBC_HIP_TRY(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices) return fail(SBC_ERR_INVALID_ARG, "device id out of range");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void *ptr = nullptr;
        SBC_HIP_TRY(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)));
        if (!ptr) return fail(SBC_ERR_HIP, "hipGetSymbolAddress gave no address for the scratch");
        g_scratch[dev] = ptr;
    }
    *out = g_scratch[dev];
    return SBC_OK;
}

}  // namespace
}  // namespace sbc

extern "C" sbc_status sbc_conv_forward(const sbc_csr *csr, const float *v,
                                       const sbc_geometry *geometry, int32_t M, const void *F,
                                       const void *W, sbc_dtype dtype, int32_t C_in,
                                       int32_t C_out, float *Y, sbc_order order, void *workspace,
                                       size_t workspace_bytes, hipStream_t stream) {
    clear_error();
    return conv_forward(csr, v, geometry, M, F, W, dtype, C_in, C_out, Y, order, workspace,
                        workspace_bytes, stream);
}

extern "C" size_t sbc_conv_forward_noalloc_max_bytes(void) { return sbc::kScratchBytes; }

extern "C" sbc_status sbc_conv_forward_noalloc(const sbc_csr *csr, const float *v,
                                               const sbc_geometry *geometry, int32_t M,
                                               const void *F, const void *W, sbc_dtype dtype,
                                               int32_t C_in, int32_t C_out, float *Y,
                                               sbc_order order, hipStream_t stream) {
    clear_error();
    SBC_TRY(check_conv_args(csr, v, geometry, M, F, W, dtype, C_in, C_out));
    SBC_TRY(check_order(order));
    const bool bf = dtype == SBC_BF16;
    const Route r = forward_route(csr->n_rows, csr->n_cols, csr->nnz_bound, M, C_in, C_out, order,
                                  bf);
    const size_t need = route_bytes(r, csr->n_rows, csr->n_cols, csr->nnz_bound, M, C_in, C_out, bf);
    if (need > kScratchBytes)
        return fail(SBC_ERR_WORKSPACE, "this forward needs " + std::to_string(need) +
                                           " bytes of temporary space; the library's static "
                                           "scratch holds " + std::to_string(kScratchBytes) +
                                           " (use sbc_conv_forward with a workspace)");
    void *ws = nullptr;
    SBC_TRY(scratch_of_current_device(&ws));
    return conv_forward(csr, v, geometry, M, F, W, dtype, C_in, C_out, Y, order, ws,
                        kScratchBytes, stream);
}

extern "C" sbc_status sbc_conv_backward(const sbc_csr *csr, const sbc_csc *csc, const float *v,
                                        const sbc_geometry *geometry, int32_t M, const void *F,
                                        const void *W, const void *dY, sbc_dtype dtype,
                                        int32_t C_in, int32_t C_out, float *dF, float *dW,
                                        sbc_order order, void *workspace, size_t workspace_bytes,
                                        hipStream_t stream) {
    clear_error();
    SBC_TRY(check_conv_args(csr, v, geometry, M, F, W, dtype, C_in, C_out));
    SBC_TRY(check_order(order));
    if (!csc || !csc->col_ptr || csc->n_cols != csr->n_cols ||
        (csr->nnz_bound > 0 && !csc->row_idx))
        return fail(SBC_ERR_INVALID_ARG, "csc is null or does not match csr");
    if (csr->nnz_bound > 0 && v && !csc->edge_perm)
        return fail(SBC_ERR_INVALID_ARG, "csc->edge_perm is needed when v is given");
    // the weighted basis normalises by row (output) sums: its transposed
    // entries take their values through edge_perm
    if (csr->nnz_bound > 0 && !v && geometry && geometry->basis == SBC_BASIS_WMONO10 &&
        !csc->edge_perm)
        return fail(SBC_ERR_INVALID_ARG, "csc->edge_perm is needed for the weighted basis");
    if (!dY && csr->n_rows > 0) return fail(SBC_ERR_INVALID_ARG, "dY is null");
    if (!aligned16(dY) || !aligned16(dF) || !aligned16(dW))
        return fail(SBC_ERR_INVALID_ARG, "dY, dF and dW must be 16-byte aligned");
    if (!dF && !dW) return SBC_OK;
    const int32_t n_out = csr->n_rows, n_in = csr->n_cols;
    const bool bf = dtype == SBC_BF16;
    const Route r = backward_route(n_out, n_in, csr->nnz_bound, M, C_in, C_out, order, bf);
    const size_t need = route_bytes(r, n_out, n_in, csr->nnz_bound, M, C_in, C_out, bf);
    if (!workspace || workspace_bytes < need)
        return fail(SBC_ERR_WORKSPACE, "workspace smaller than sbc_conv_workspace_size()");
    if (route_fused(r, M, C_in, C_out, bf))
        return fused_backward(csr, csc, v, geometry, M, F, W, dY, bf, C_in, C_out, dF, dW,
                              workspace, stream);

    ConvWs ws = carve_route(workspace, r, n_out, n_in, csr->nnz_bound, M, C_in, C_out, nullptr);
    // values of the transposed entries: through edge_perm, or (with no
    // edge_perm, so v is null) evaluated in the transpose's own order into
    // ws.v once the CSR-ordered values are no longer needed
    const float *vv = v;
    const int32_t *perm_t = csc->edge_perm;
    auto values_t = [&]() -> sbc_status {
        if (perm_t) return SBC_OK;
        SBC_TRY(basis_eval_t_launch(csc, csr->nnz_bound, geometry, ws.v, stream));
        vv = ws.v;
        return SBC_OK;
    };
    if (!vv && (r == kBwdG || perm_t)) {
        SBC_TRY(basis_eval_launch(csr, geometry, ws.v, stream));
        vv = ws.v;
    }
    const int64_t K1 = (int64_t)M * C_in, K2 = (int64_t)M * C_out;
    if (r == kBwdG) {
        SBC_TRY(spmm(n_out, csr->row_ptr, csr->col_idx, nullptr, vv, M, F, bf, C_in, false,
                     csr->nnz_bound, ws.inter, stream, "bwd_spmm"));
        if (dW)  // dW [M*C_in, C_out] = G^T dY
            SBC_TRY(gemm(ws.inter, false, 1, K1, dY, bf, C_out, 1, dW, C_out, 1, (int32_t)K1,
                         C_out, n_out, ws.partial, stream, "bwd_gemm_dw"));
        if (dF) {  // dG = dY W_flat^T, then dF = N^T dG
            SBC_TRY(gemm(dY, bf, C_out, 1, W, bf, 1, C_out, ws.inter2, K1, 1, n_out, (int32_t)K1,
                         C_out, ws.partial, stream, "bwd_gemm_dg"));
            SBC_TRY(values_t());
            SBC_TRY(spmm(n_in, csc->col_ptr, csc->row_idx, perm_t, vv, M, ws.inter2, false, C_in,
                         true, csr->nnz_bound, dF, stream, "bwd_spmm_t"));
        }
    } else {
        SBC_TRY(values_t());
        SBC_TRY(spmm(n_in, csc->col_ptr, csc->row_idx, perm_t, vv, M, dY, bf, C_out, false,
                     csr->nnz_bound, ws.inter, stream, "bwd_spmm_t_expand"));
        if (dF) {  // Wt [M, C_out, C_in]; dF = D Wt
            SBC_TRY(permute_w(W, bf, M, C_in, C_out, (int64_t)C_out * C_in, 1, C_in, ws.wperm,
                              stream));
            SBC_TRY(gemm(ws.inter, false, K2, 1, ws.wperm, false, C_in, 1, dF, C_in, 1, n_in,
                         C_in, K2, ws.partial, stream, "bwd_gemm_df"));
        }
        if (dW) {  // dW' [C_in, M*C_out] = F^T D, then back to [M, C_in, C_out]
            SBC_TRY(gemm(F, bf, 1, C_in, ws.inter, false, K2, 1, ws.dwperm, K2, 1, C_in,
                         (int32_t)K2, n_in, ws.partial, stream, "bwd_gemm_dw_t"));
            SBC_TRY(permute_w_back(ws.dwperm, M, C_in, C_out, dW, stream));
        }
    }
    return SBC_OK;
}

// ---------------------------------------------------------------- decay rates
namespace sbc {
namespace {

// dlambda[m] = <dW'_m, W_m> over the C_in x C_out block of m: one block per m,
// float64 sums over a fixed thread assignment, then a fixed-order tree.
template <typename WT>
__global__ void __launch_bounds__(256)
    decay_dot_kernel(const float *__restrict__ dWp, const WT *__restrict__ W, int64_t per_m,
                     float *__restrict__ dlambda) {
    __shared__ double s[256];
    const int64_t base = (int64_t)blockIdx.x * per_m;
    double acc = 0.0;
    for (int64_t x = threadIdx.x; x < per_m; x += 256) {
        float w;
        if constexpr (sizeof(WT) == 2)
            w = __uint_as_float((uint32_t)W[base + x] << 16);
        else
            w = W[base + x];
        acc += (double)dWp[base + x] * (double)w;
    }
    s[threadIdx.x] = acc;
    __syncthreads();
    for (int d = 128; d >= 1; d >>= 1) {
        if ((int)threadIdx.x < d) s[threadIdx.x] += s[threadIdx.x + d];
        __syncthreads();
    }
    if (threadIdx.x == 0) dlambda[blockIdx.x] = (float)s[0];
}

struct DecayWs {
    float *v, *G, *dWp, *partial;
};

DecayWs carve_decay(void *base, int32_t n, int64_t nnz, int32_t M, int32_t Ci, int32_t Co,
                    size_t *bytes) {
    Carver cv(base);
    DecayWs w;
    w.v = cv.take<float>((size_t)(nnz > 0 ? nnz : 0) * M);
    w.G = cv.take<float>((size_t)n * M * Ci);
    w.dWp = cv.take<float>((size_t)M * Ci * Co);
    w.partial = cv.take<float>(gemm_workspace_floats(M * Ci, Co, n));
    if (bytes) *bytes = cv.used;
    return w;
}

}  // namespace
}  // namespace sbc

extern "C" size_t sbc_decay_gradient_workspace_size(int32_t n, int64_t nnz_bound, int32_t M,
                                                    int32_t C_in, int32_t C_out,
                                                    sbc_dtype dtype) {
    if (n < 0 || nnz_bound < 0 || M <= 0 || C_in <= 0 || C_out <= 0) return 0;
    size_t bytes = 0;
    carve_decay(nullptr, n, nnz_bound, M, C_in, C_out, &bytes);
    // the fused D-route: its own workspace, then dW'
    const size_t fused = fused_workspace_bytes(M, C_in, C_out, n, nnz_bound) +
                         align_up((size_t)M * C_in * C_out * 4);
    return fused_backward_available(M, C_in, C_out, dtype == SBC_BF16) && fused > bytes ? fused
                                                                                        : bytes;
}

extern "C" sbc_status sbc_conv_decay_gradient(const sbc_csr *csr, const sbc_csc *csc,
                                              const sbc_geometry *geometry, int32_t M,
                                              const void *F, const void *W, const void *dY,
                                              sbc_dtype dtype, int32_t C_in, int32_t C_out,
                                              float *dlambda, void *workspace,
                                              size_t workspace_bytes, hipStream_t stream) {
    clear_error();
    SBC_TRY(check_conv_args(csr, nullptr, geometry, M, F, W, dtype, C_in, C_out));
    if (geometry->basis != SBC_BASIS_EVENT_DECAYS)
        return fail(SBC_ERR_INVALID_ARG, "the decay gradient needs SBC_BASIS_EVENT_DECAYS");
    if (!dlambda || (csr->n_rows > 0 && !dY))
        return fail(SBC_ERR_INVALID_ARG, "dY or dlambda is null");
    if (csc && (!csc->col_ptr || csc->n_cols != csr->n_cols ||
                (csr->nnz_bound > 0 && !csc->row_idx)))
        return fail(SBC_ERR_INVALID_ARG, "csc does not match csr");
    const int32_t n = csr->n_rows;
    const bool bf = dtype == SBC_BF16;
    const size_t need = sbc_decay_gradient_workspace_size(n, csr->nnz_bound, M, C_in, C_out, dtype);
    if (!workspace || workspace_bytes < need)
        return fail(SBC_ERR_WORKSPACE, "workspace smaller than sbc_decay_gradient_workspace_size()");
    if (n == 0) return fill_i32(reinterpret_cast<int32_t *>(dlambda), 0, M, stream);
    float *dWp;
    if (csc && fused_backward_available(M, C_in, C_out, bf)) {
        // D' = N'^T dY gathered with the derivative values, dW' = F^T D' (dF skipped)
        const int32_t np = n > csr->n_cols ? n : csr->n_cols;
        dWp = reinterpret_cast<float *>(static_cast<char *>(workspace) +
                                        fused_workspace_bytes(M, C_in, C_out, np, csr->nnz_bound));
        SBC_TRY(fused_backward(csr, csc, nullptr, geometry, M, F, W, dY, bf, C_in, C_out, nullptr,
                               dWp, workspace, stream, true));
    } else {
        // v' = d p / d lambda, G' = N' F, dW' = G'^T dY
        DecayWs ws = carve_decay(workspace, n, csr->nnz_bound, M, C_in, C_out, nullptr);
        SBC_TRY(decay_derivative_launch(csr, geometry, ws.v, stream));
        SBC_TRY(spmm(n, csr->row_ptr, csr->col_idx, nullptr, ws.v, M, F, bf, C_in, false,
                     csr->nnz_bound, ws.G, stream, "decay_spmm"));
        const int64_t K1 = (int64_t)M * C_in;
        SBC_TRY(gemm(ws.G, false, 1, K1, dY, bf, C_out, 1, ws.dWp, C_out, 1, (int32_t)K1, C_out,
                     n, ws.partial, stream, "decay_gemm"));
        dWp = ws.dWp;
    }
    trace_before("decay_dot", stream);
    const int64_t per_m = (int64_t)C_in * C_out;
    if (bf)
        hipLaunchKernelGGL(decay_dot_kernel<uint16_t>, dim3(M), dim3(256), 0, stream, dWp,
                           static_cast<const uint16_t *>(W), per_m, dlambda);
    else
        hipLaunchKernelGGL(decay_dot_kernel<float>, dim3(M), dim3(256), 0, stream, dWp,
                           static_cast<const float *>(W), per_m, dlambda);
    SBC_LAUNCH_CHECK();
    trace_after("decay_dot", stream);
    return SBC_OK;
}
