// Subsampling of point clouds (Section 3.1, "Subsampling", and the
// supplementary algorithms): iterative farthest points, its approximation with
// distance updates limited to the ball neighbourhood of each taken point, and
// rejection sampling (taking, in input order, every point no earlier taken
// point has in its ball), alone or followed by the approximation.
//
// One workgroup per cloud, with the cloud's squared distances and sampling
// states in LDS:
//   - rejection sampling is the lexicographically first maximal independent
//     set of the ball graph; it is found in rounds: an undecided point whose
//     earlier neighbours are all decided is taken if none of them was taken,
//     else rejected.  The lowest undecided point always decides, so the rounds
//     end, and a decision depends only on final states, so the result is the
//     sequential one whatever the timing;
//   - farthest points: each step is an argmax over the points not yet taken
//     (ties to the lowest index), then the distances are lowered to the new
//     point (all of them, or its ball neighbours).
// Squared distances are float32 in the canonical form of the neighbour search,
// so every choice is exact.
#include "common.hpp"

namespace sbc {
namespace {

constexpr int kSampThreads = 512;
constexpr int kSampMax = 8192;  // points per cloud held in LDS

// the canonical form, with no contraction of the products into the sums
__device__ __forceinline__ float sq_dist(const float *__restrict__ x, int64_t a, int64_t b) {
#pragma clang fp contract(off)
    const float dx = x[3 * a] - x[3 * b], dy = x[3 * a + 1] - x[3 * b + 1],
                dz = x[3 * a + 2] - x[3 * b + 2];
    return (dx * dx + dy * dy) + dz * dz;
}

struct SampleArgs {
    const float *x;
    const int32_t *splits;
    const int32_t *row_ptr, *col_idx;  // in-place ball CSR (may be null for exact IFP)
    int32_t method, per_cloud;
    const int32_t *out_splits;         // (null in the counting pass of rejection sampling)
    int32_t *out_idx, *counts;
    float *dmin2;
};

// kWrite false: the counting pass (each cloud's number of outputs; rejection
// sampling alone decides its points here to count them); kWrite true: the
// sampling, writing the indices at out_splits[b] and the squared distances.
template <bool kWrite>
__global__ void __launch_bounds__(kSampThreads) sample_kernel(SampleArgs A) {
    __shared__ float s_d[kSampMax];
    __shared__ uint8_t s_st[kSampMax];  // 0 undecided, 1 taken, 2 rejected
    __shared__ float s_bv[kSampThreads];
    __shared__ int32_t s_bi[kSampThreads];
    __shared__ int32_t s_cnt;
    const int tid = threadIdx.x;
    const int32_t b = blockIdx.x;
    const int32_t s = A.splits[b], n = A.splits[b + 1] - s;
    const bool rej = A.method == SBC_SAMPLE_REJECTION || A.method == SBC_SAMPLE_APPROX_IFP_REJECTION;
    const bool approx = A.method != SBC_SAMPLE_IFP;
    if (n > kSampMax || n < 0) {  // beyond the LDS state (the caller's bound): no outputs
        if (!kWrite && tid == 0) A.counts[b] = 0;
        return;
    }
    if (!kWrite && A.method != SBC_SAMPLE_REJECTION) {
        if (tid == 0) A.counts[b] = A.per_cloud < n ? A.per_cloud : n;
        return;
    }
    for (int32_t j = tid; j < n; j += kSampThreads) {
        s_d[j] = INFINITY;
        s_st[j] = 0;
    }
    if (tid == 0) s_cnt = 0;
    __syncthreads();
    if (rej) {
        // rounds of the first maximal independent set of the ball graph
        bool more = true;
        while (more) {
            bool undecided = false;
            for (int32_t j = tid; j < n; j += kSampThreads) {
                if (s_st[j] != 0) continue;
                bool pending = false, hit = false;
                const int32_t e1 = A.row_ptr[s + j + 1];
                for (int32_t e = A.row_ptr[s + j]; e < e1; ++e) {
                    const int32_t k = A.col_idx[e] - s;
                    if (k < 0 || k >= j) continue;  // later points (and any outside the cloud)
                    const uint8_t st = s_st[k];
                    if (st == 1) { hit = true; break; }
                    if (st == 0) pending = true;
                }
                if (hit) s_st[j] = 2;
                else if (!pending) s_st[j] = 1;
                else undecided = true;
            }
            more = __syncthreads_or(undecided);
        }
        // distances to the nearest taken neighbour; count the taken points
        int32_t mine = 0;
        for (int32_t j = tid; j < n; j += kSampThreads) {
            float d = INFINITY;
            const int32_t e1 = A.row_ptr[s + j + 1];
            for (int32_t e = A.row_ptr[s + j]; e < e1; ++e) {
                const int32_t k = A.col_idx[e] - s;
                if (k >= 0 && k < n && s_st[k] == 1) {
                    const float q = sq_dist(A.x, (int64_t)s + k, (int64_t)s + j);
                    d = q < d ? q : d;
                }
            }
            s_d[j] = d;
            mine += s_st[j] == 1 ? 1 : 0;
        }
        atomicAdd(&s_cnt, mine);  // an integer count: order-free
        __syncthreads();
    }
    const int32_t taken = s_cnt;
    const int32_t total = A.method == SBC_SAMPLE_REJECTION ? taken
                          : (A.per_cloud < n ? A.per_cloud : n);
    if (!kWrite) {
        if (tid == 0) A.counts[b] = total;
        return;
    }
    const int32_t base = A.out_splits[b];
    int32_t pos = 0;
    if (rej) {
        // the taken points first, in input order (a workgroup scan over chunks)
        const int32_t cap = taken < total ? taken : total;
        for (int32_t c0 = 0; c0 < n; c0 += kSampThreads) {
            const int32_t j = c0 + tid;
            const int32_t f = (j < n && s_st[j] == 1) ? 1 : 0;
            s_bi[tid] = f;
            __syncthreads();
            for (int d = 1; d < kSampThreads; d <<= 1) {
                const int32_t y = tid >= d ? s_bi[tid - d] : 0;
                __syncthreads();
                s_bi[tid] += y;
                __syncthreads();
            }
            const int32_t rank = pos + s_bi[tid] - f;
            if (f && rank < cap) A.out_idx[base + rank] = s + j;
            pos += s_bi[kSampThreads - 1];
            __syncthreads();
        }
        pos = cap;
    }
    for (int32_t it = pos; it < total; ++it) {
        // argmax of the distances over the points not yet taken, ties to the
        // lowest index (a taken point is never taken again, which matters
        // once every remaining distance is 0: coincident points)
        float bv = -1.f;
        int32_t bi = 0;
        for (int32_t j = tid; j < n; j += kSampThreads) {
            const float d = s_d[j];
            if (s_st[j] != 1 && d > bv) { bv = d; bi = j; }
        }
        s_bv[tid] = bv;
        s_bi[tid] = bi;
        __syncthreads();
        for (int d = kSampThreads / 2; d >= 1; d >>= 1) {
            if (tid < d) {
                const float v2 = s_bv[tid + d];
                const int32_t i2 = s_bi[tid + d];
                if (v2 > s_bv[tid] || (v2 == s_bv[tid] && i2 < s_bi[tid])) {
                    s_bv[tid] = v2;
                    s_bi[tid] = i2;
                }
            }
            __syncthreads();
        }
        const int32_t sel = s_bi[0];
        if (tid == 0) {
            A.out_idx[base + it] = s + sel;
            s_st[sel] = 1;  // read again only after the barrier closing this step
        }
        if (approx) {
            const int32_t e0 = A.row_ptr[s + sel], e1 = A.row_ptr[s + sel + 1];
            for (int32_t e = e0 + tid; e < e1; e += kSampThreads) {
                const int32_t k = A.col_idx[e] - s;
                if (k >= 0 && k < n) {
                    const float q = sq_dist(A.x, (int64_t)s + k, (int64_t)s + sel);
                    if (q < s_d[k]) s_d[k] = q;
                }
            }
        } else {
            for (int32_t j = tid; j < n; j += kSampThreads) {
                const float q = sq_dist(A.x, (int64_t)s + j, (int64_t)s + sel);
                if (q < s_d[j]) s_d[j] = q;
            }
        }
        __syncthreads();
    }
    if (A.dmin2)
        for (int32_t j = tid; j < n; j += kSampThreads) A.dmin2[s + j] = s_d[j];
}

}  // namespace
}  // namespace sbc

using namespace sbc;

extern "C" size_t sbc_sampling_workspace_size(int32_t n_batch) {
    if (n_batch < 0) return 0;
    return align_up((size_t)n_batch * 4) + align_up(16) + scan_workspace_bytes(n_batch);
}

extern "C" sbc_status sbc_sample_points(const float *x, const int32_t *splits, int32_t n_batch,
                                        int32_t n_points, int32_t max_cloud,
                                        const sbc_csr *ball, sbc_sampling method,
                                        int32_t per_cloud, int32_t *out_idx,
                                        int32_t *out_splits, float *dmin2, void *workspace,
                                        size_t workspace_bytes, hipStream_t stream) {
    clear_error();
    if (n_batch < 1 || !splits || !out_splits || n_points < 0)
        return fail(SBC_ERR_INVALID_ARG, "n_batch must be >= 1 with splits and out_splits");
    if (method != SBC_SAMPLE_IFP && method != SBC_SAMPLE_APPROX_IFP &&
        method != SBC_SAMPLE_APPROX_IFP_REJECTION && method != SBC_SAMPLE_REJECTION)
        return fail(SBC_ERR_INVALID_ARG, "unknown sampling method");
    if (method != SBC_SAMPLE_REJECTION && per_cloud < 0)
        return fail(SBC_ERR_INVALID_ARG, "per_cloud must be >= 0");
    if (max_cloud < 0 || max_cloud > kSampMax)
        return fail(SBC_ERR_UNSUPPORTED, "clouds of at most 8192 points");
    if (n_points > 0 && (!x || !out_idx)) return fail(SBC_ERR_INVALID_ARG, "x or out_idx is null");
    if (method != SBC_SAMPLE_IFP &&
        (!ball || !ball->row_ptr || ball->n_rows != n_points || ball->n_cols != n_points ||
         (ball->nnz_bound > 0 && !ball->col_idx)))
        return fail(SBC_ERR_INVALID_ARG, "the in-place ball pattern of the points is needed");
    const size_t need = sbc_sampling_workspace_size(n_batch);
    if (!workspace || workspace_bytes < need)
        return fail(SBC_ERR_WORKSPACE, "workspace smaller than sbc_sampling_workspace_size()");
    Carver cv(workspace);
    int32_t *counts = cv.take<int32_t>(n_batch);
    int64_t *total = cv.take<int64_t>(2);
    void *scan_ws = cv.take<char>(scan_workspace_bytes(n_batch));
    SampleArgs A{};
    A.x = x;
    A.splits = splits;
    A.row_ptr = ball ? ball->row_ptr : nullptr;
    A.col_idx = ball ? ball->col_idx : nullptr;
    A.method = method;
    A.per_cloud = per_cloud;
    A.out_idx = out_idx;
    A.counts = counts;
    A.dmin2 = nullptr;
    // counts per cloud (rejection sampling runs once here to count), bounds,
    // then the sampling with its writes
    trace_before("sample_count", stream);
    hipLaunchKernelGGL(sample_kernel<false>, dim3(n_batch), dim3(kSampThreads), 0, stream, A);
    SBC_LAUNCH_CHECK();
    trace_after("sample_count", stream);
    SBC_TRY(exclusive_scan_i32(counts, out_splits, n_batch, total, scan_ws, stream));
    A.out_splits = out_splits;
    A.dmin2 = dmin2;
    trace_before("sample", stream);
    hipLaunchKernelGGL(sample_kernel<true>, dim3(n_batch), dim3(kSampThreads), 0, stream, A);
    SBC_LAUNCH_CHECK();
    trace_after("sample", stream);
    return SBC_OK;
}
