// Device-wide exclusive prefix sums, fills and small segmented sorts.
//
// Scan: up to 8192 items, one block walks the array.  Beyond, a blocked
// scan: each block of 256 threads owns 1024 consecutive items (4 per thread)
// and publishes its total (int64, so edge totals beyond 2^31 are detected
// exactly); a second kernel's blocks each add up the preceding totals
// themselves and rescan their items (for very long arrays the totals are
// scanned recursively instead).
#include <climits>

#include "common.hpp"

namespace sbc {
namespace {

constexpr int kThreads = 256;
constexpr int kItems = 4;
constexpr int kPerBlock = kThreads * kItems;  // 1024

// Inclusive scan of one int64 per thread across a 256-thread block.
__device__ int64_t block_inclusive_scan(int64_t x, int64_t *lds /*[4]*/, int64_t *block_total) {
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        int64_t y = __shfl_up(x, d, 64);
        if (lane >= d) x += y;
    }
    if (lane == 63) lds[wave] = x;
    __syncthreads();
    int64_t before = 0, total = 0;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) {
        int64_t s = lds[w];
        if (w < wave) before += s;
        total += s;
    }
    __syncthreads();
    *block_total = total;
    return x + before;
}

// Block totals; with in2 (two arrays of n items scanned in one launch) blocks
// nb .. 2 nb - 1 take in2, and sums holds the first array's totals, then the
// second's.
template <typename T>
__global__ void __launch_bounds__(kThreads)
    block_sums_kernel(const T *in, int64_t n, int64_t *sums, const T *in2, int64_t nb) {
    __shared__ int64_t lds[kThreads / 64];
    const bool second = in2 && (int64_t)blockIdx.x >= nb;
    if (second) in = in2;
    const int64_t blk = second ? (int64_t)blockIdx.x - nb : (int64_t)blockIdx.x;
    const int64_t base = blk * kPerBlock + (int64_t)threadIdx.x * kItems;
    int64_t s = 0;
#pragma unroll
    for (int k = 0; k < kItems; ++k)
        if (base + k < n) s += (int64_t)in[base + k];
    int64_t total;
    block_inclusive_scan(s, lds, &total);
    if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

// Exclusive scan of `in` with per-block offsets (offsets == nullptr: zero),
// written to `out`.  OutT int32 saturates at INT_MAX.
template <typename InT, typename OutT>
__global__ void __launch_bounds__(kThreads)
    block_scan_kernel(const InT *in, int64_t n, const int64_t *offsets, OutT *out,
                      int64_t *total64, bool write_total, OutT *out2) {
    __shared__ int64_t lds[kThreads / 64];
    const int64_t base = (int64_t)blockIdx.x * kPerBlock + (int64_t)threadIdx.x * kItems;
    int64_t v[kItems];
    int64_t s = 0;
#pragma unroll
    for (int k = 0; k < kItems; ++k) {
        v[k] = (base + k < n) ? (int64_t)in[base + k] : 0;
        s += v[k];
    }
    int64_t total;
    int64_t incl = block_inclusive_scan(s, lds, &total);
    int64_t run = incl - s + (offsets ? offsets[blockIdx.x] : 0);
#pragma unroll
    for (int k = 0; k < kItems; ++k) {
        if (base + k < n) {
            OutT o;
            if (sizeof(OutT) == 4)
                o = (OutT)(run > (int64_t)INT_MAX ? (int64_t)INT_MAX : run);
            else
                o = (OutT)run;
            out[base + k] = o;
            if (out2) out2[base + k] = o;
        }
        run += v[k];
    }
    // the thread holding item n-1 (or, past it, the block's last thread) knows
    // the grand total
    if (write_total && blockIdx.x == gridDim.x - 1 && threadIdx.x == kThreads - 1) {
        int64_t grand = (offsets ? offsets[blockIdx.x] : 0) + total;
        OutT o;
        if (sizeof(OutT) == 4)
            o = (OutT)(grand > (int64_t)INT_MAX ? (int64_t)INT_MAX : grand);
        else
            o = (OutT)grand;
        out[n] = o;
        if (out2) out2[n] = o;
        if (total64) *total64 = grand;
    }
}

// Single-block scan for short arrays: 1024 threads walk the array in chunks
// of 1024 x kSmallItems, carrying the running total; the next chunk is loaded
// while the current one is scanned.  out2 (optional) receives a copy.
constexpr int kSmallThreads = 1024;
constexpr int kSmallItems = 8;
constexpr int64_t kSmallMax = 8192;
// Up to this many blocks, each block sums the preceding block totals itself.
constexpr int64_t kSelfOffsetBlocks = 4096;

__global__ void __launch_bounds__(kSmallThreads)
    small_scan_kernel(const int32_t *__restrict__ in, int64_t n, int32_t *__restrict__ out,
                      int32_t *__restrict__ out2, int64_t *__restrict__ total64) {
    __shared__ int64_t wsum[kSmallThreads / 64];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    constexpr int64_t chunk = (int64_t)kSmallThreads * kSmallItems;
    int64_t carry = 0;
    int32_t cur[kSmallItems];
    int64_t base = (int64_t)threadIdx.x * kSmallItems;
#pragma unroll
    for (int k = 0; k < kSmallItems; ++k) cur[k] = (base + k < n) ? in[base + k] : 0;
    for (int64_t c0 = 0; c0 < n; c0 += chunk) {
        int32_t nxt[kSmallItems];
        const int64_t nb = c0 + chunk + (int64_t)threadIdx.x * kSmallItems;
#pragma unroll
        for (int k = 0; k < kSmallItems; ++k) nxt[k] = (nb + k < n) ? in[nb + k] : 0;
        int64_t s = 0;
#pragma unroll
        for (int k = 0; k < kSmallItems; ++k) s += cur[k];
        int64_t x = s;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            int64_t y = __shfl_up(x, d, 64);
            if (lane >= d) x += y;
        }
        if (lane == 63) wsum[wave] = x;
        __syncthreads();
        int64_t before = 0, tot = 0;
#pragma unroll
        for (int w = 0; w < kSmallThreads / 64; ++w) {
            const int64_t v = wsum[w];
            before += (w < wave) ? v : 0;
            tot += v;
        }
        __syncthreads();
        int64_t run = carry + before + x - s;
        const int64_t b0 = c0 + (int64_t)threadIdx.x * kSmallItems;
#pragma unroll
        for (int k = 0; k < kSmallItems; ++k) {
            if (b0 + k < n) {
                const int32_t o = (int32_t)(run > (int64_t)INT_MAX ? (int64_t)INT_MAX : run);
                out[b0 + k] = o;
                if (out2) out2[b0 + k] = o;
            }
            run += cur[k];
        }
        carry += tot;
#pragma unroll
        for (int k = 0; k < kSmallItems; ++k) cur[k] = nxt[k];
    }
    if (threadIdx.x == 0) {
        const int32_t o = (int32_t)(carry > (int64_t)INT_MAX ? (int64_t)INT_MAX : carry);
        out[n] = o;
        if (out2) out2[n] = o;
        if (total64) *total64 = carry;
    }
}

// Second pass of the two-kernel scan: block b first adds up the totals of
// blocks 0..b-1 (all 256 threads, then a block reduction; the order is fixed),
// then scans its own items with that offset.  With in2 (a second array of n
// items), blocks nb .. 2 nb - 1 scan in2 into outb with the second array's
// totals (sums + nb), and its grand total goes to totalb.
__global__ void __launch_bounds__(kThreads)
    self_offset_scan_kernel(const int32_t *__restrict__ in, int64_t n,
                            const int64_t *__restrict__ sums, int32_t *__restrict__ out,
                            int32_t *__restrict__ out2, int64_t *__restrict__ total64,
                            const int32_t *__restrict__ in2, int32_t *__restrict__ outb,
                            int64_t *__restrict__ totalb, int64_t nb) {
    __shared__ int64_t lds[kThreads / 64];
    __shared__ int64_t red[kThreads];
    const bool second = in2 && (int64_t)blockIdx.x >= nb;
    const int64_t blk = second ? (int64_t)blockIdx.x - nb : (int64_t)blockIdx.x;
    const int64_t last_blk = in2 ? nb - 1 : (int64_t)gridDim.x - 1;
    if (second) {
        in = in2;
        out = outb;
        out2 = nullptr;
        total64 = totalb;
        sums += nb;
    }
    int64_t part = 0;
    for (int64_t q = threadIdx.x; q < blk; q += kThreads) part += sums[q];
    red[threadIdx.x] = part;
    __syncthreads();
    for (int w = kThreads / 2; w > 0; w >>= 1) {
        if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
        __syncthreads();
    }
    const int64_t offset = red[0];
    const int64_t base = blk * kPerBlock + (int64_t)threadIdx.x * kItems;
    int64_t v[kItems];
    int64_t s = 0;
#pragma unroll
    for (int k = 0; k < kItems; ++k) {
        v[k] = (base + k < n) ? (int64_t)in[base + k] : 0;
        s += v[k];
    }
    int64_t total;
    const int64_t incl = block_inclusive_scan(s, lds, &total);
    int64_t run = incl - s + offset;
#pragma unroll
    for (int k = 0; k < kItems; ++k) {
        if (base + k < n) {
            const int32_t o = (int32_t)(run > (int64_t)INT_MAX ? (int64_t)INT_MAX : run);
            out[base + k] = o;
            if (out2) out2[base + k] = o;
        }
        run += v[k];
    }
    if (blk == last_blk && threadIdx.x == kThreads - 1) {
        const int64_t grand = offset + total;
        const int32_t o = (int32_t)(grand > (int64_t)INT_MAX ? (int64_t)INT_MAX : grand);
        out[n] = o;
        if (out2) out2[n] = o;
        if (total64) *total64 = grand;
    }
}

// In-place exclusive scan of n int64 values; `ws` holds the recursion's sums.
sbc_status scan_i64_inplace(int64_t *a, int64_t n, char *ws, hipStream_t stream) {
    if (n <= 0) return SBC_OK;
    const int64_t nb = (n + kPerBlock - 1) / kPerBlock;
    if (nb == 1) {
        hipLaunchKernelGGL((block_scan_kernel<int64_t, int64_t>), dim3(1), dim3(kThreads), 0,
                           stream, a, n, (const int64_t *)nullptr, a, (int64_t *)nullptr, false,
                           (int64_t *)nullptr);
        SBC_LAUNCH_CHECK();
        return SBC_OK;
    }
    int64_t *sums = reinterpret_cast<int64_t *>(ws);
    char *rest = ws + align_up(nb * sizeof(int64_t));
    hipLaunchKernelGGL((block_sums_kernel<int64_t>), dim3((unsigned)nb), dim3(kThreads), 0, stream,
                       a, n, sums, (const int64_t *)nullptr, nb);
    SBC_LAUNCH_CHECK();
    SBC_TRY(scan_i64_inplace(sums, nb, rest, stream));
    hipLaunchKernelGGL((block_scan_kernel<int64_t, int64_t>), dim3((unsigned)nb), dim3(kThreads),
                       0, stream, a, n, (const int64_t *)sums, a, (int64_t *)nullptr, false,
                       (int64_t *)nullptr);
    SBC_LAUNCH_CHECK();
    return SBC_OK;
}

size_t scan_i64_ws(int64_t n) {
    size_t bytes = 0;
    while (n > kPerBlock) {
        int64_t nb = (n + kPerBlock - 1) / kPerBlock;
        bytes += align_up(nb * sizeof(int64_t));
        n = nb;
    }
    return bytes;
}

__global__ void fill_kernel(int32_t *p, int32_t value, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = value;
}

// One thread per entry p < min(ptr[n_segments], n_bound): its segment is
// seg_of[p], and its rank is the number of keys of that segment below its own
// (keys are distinct within a segment), so it moves to ptr[seg] + rank.  A
// segment of length L costs L^2 key reads in all, spread over L threads; the
// segments here are neighbourhood columns and pixel lists, a few tens long.
// Ranks stay inside the segment even for repeated keys (an entry is never
// counted below itself), so every write is in bounds.
__global__ void __launch_bounds__(256)
    rank_sort_kernel(const int32_t *__restrict__ ptr, int32_t n_segments,
                     const int32_t *__restrict__ seg_of, int64_t n_bound,
                     const int32_t *__restrict__ key_in, const int32_t *__restrict__ val_in,
                     int32_t *__restrict__ key_out, int32_t *__restrict__ val_out) {
    int64_t n = ptr[n_segments];
    n = n < n_bound ? n : n_bound;
    for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < n;
         p += (int64_t)gridDim.x * blockDim.x) {
        const int32_t sg = seg_of[p];
        const int32_t s = ptr[sg], t = ptr[sg + 1];
        const int32_t k = key_in[p];
        int32_t rank = 0;
        for (int32_t b = s; b < t; ++b) rank += key_in[b] < k ? 1 : 0;
        key_out[s + rank] = k;
        if (val_out) val_out[s + rank] = val_in[p];
    }
}

}  // namespace

size_t scan_workspace_bytes(int64_t n) {
    int64_t nb = (n + kPerBlock - 1) / kPerBlock;
    return align_up((nb > 0 ? nb : 1) * sizeof(int64_t)) + scan_i64_ws(nb);
}

sbc_status fill_i32(int32_t *p, int32_t value, int64_t n, hipStream_t stream) {
    if (n <= 0) return SBC_OK;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(fill_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, p, value, n);
    SBC_LAUNCH_CHECK();
    return SBC_OK;
}

sbc_status exclusive_scan_i32(const int32_t *counts, int32_t *out, int64_t n, int64_t *total64,
                              void *ws, hipStream_t stream, int32_t *out2) {
    if (n <= kSmallMax) {
        hipLaunchKernelGGL(small_scan_kernel, dim3(1), dim3(kSmallThreads), 0, stream, counts,
                           n > 0 ? n : 0, out, out2, total64);
        SBC_LAUNCH_CHECK();
        return SBC_OK;
    }
    const int64_t nb = (n + kPerBlock - 1) / kPerBlock;
    char *w = static_cast<char *>(ws);
    int64_t *sums = reinterpret_cast<int64_t *>(w);
    char *rest = w + align_up(nb * sizeof(int64_t));
    hipLaunchKernelGGL((block_sums_kernel<int32_t>), dim3((unsigned)nb), dim3(kThreads), 0, stream,
                       counts, n, sums, (const int32_t *)nullptr, nb);
    SBC_LAUNCH_CHECK();
    if (nb <= kSelfOffsetBlocks) {
        hipLaunchKernelGGL(self_offset_scan_kernel, dim3((unsigned)nb), dim3(kThreads), 0, stream,
                           counts, n, (const int64_t *)sums, out, out2, total64,
                           (const int32_t *)nullptr, (int32_t *)nullptr, (int64_t *)nullptr, nb);
        SBC_LAUNCH_CHECK();
        return SBC_OK;
    }
    SBC_TRY(scan_i64_inplace(sums, nb, rest, stream));
    hipLaunchKernelGGL((block_scan_kernel<int32_t, int32_t>), dim3((unsigned)nb), dim3(kThreads),
                       0, stream, counts, n, (const int64_t *)sums, out, total64, true, out2);
    SBC_LAUNCH_CHECK();
    return SBC_OK;
}

size_t scan2_workspace_bytes(int64_t n) {
    const int64_t nb = (n + kPerBlock - 1) / kPerBlock;
    const size_t pair = align_up((nb > 0 ? 2 * nb : 1) * sizeof(int64_t));
    const size_t one = scan_workspace_bytes(n);
    return pair > one ? pair : one;
}

sbc_status exclusive_scan2_i32(const int32_t *a, int32_t *a_out, const int32_t *b,
                               int32_t *b_out, int64_t n, int64_t *a_total64,
                               int64_t *b_total64, void *ws, hipStream_t stream) {
    const int64_t nb = (n + kPerBlock - 1) / kPerBlock;
    if (n <= kSmallMax || nb > kSelfOffsetBlocks) {
        SBC_TRY(exclusive_scan_i32(a, a_out, n, a_total64, ws, stream));
        return exclusive_scan_i32(b, b_out, n, b_total64, ws, stream);
    }
    int64_t *sums = static_cast<int64_t *>(ws);
    hipLaunchKernelGGL((block_sums_kernel<int32_t>), dim3((unsigned)(2 * nb)), dim3(kThreads), 0,
                       stream, a, n, sums, b, nb);
    SBC_LAUNCH_CHECK();
    hipLaunchKernelGGL(self_offset_scan_kernel, dim3((unsigned)(2 * nb)), dim3(kThreads), 0, stream,
                       a, n, (const int64_t *)sums, a_out, (int32_t *)nullptr, a_total64, b, b_out,
                       b_total64, nb);
    SBC_LAUNCH_CHECK();
    return SBC_OK;
}

sbc_status segmented_sort_pairs(const int32_t *ptr, int32_t n_segments, const int32_t *seg_of,
                                int64_t n_bound, const int32_t *key_in, const int32_t *val_in,
                                int32_t *key_out, int32_t *val_out, hipStream_t stream) {
    if (n_segments <= 0 || n_bound <= 0) return SBC_OK;
    int64_t blocks = (n_bound + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(rank_sort_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, ptr,
                       n_segments, seg_of, n_bound, key_in, val_in, key_out, val_out);
    SBC_LAUNCH_CHECK();
    return SBC_OK;
}

}  // namespace sbc
