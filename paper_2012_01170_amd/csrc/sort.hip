// Stable least-significant-digit radix sort of (key, value) int32 pairs, with
// no global atomics: each pass counts digits per block in LDS, scans the
// [digit][block] counts across the device, and scatters every block's items
// to their digit's range in order.  Within a block an item's place among
// equal digits comes from wave ballots (lanes with the same digit in the
// same 64-item round) and per-wave running counts, so equal digits keep their
// input order and the sort is stable; the result does not depend on
// scheduling.
//
// Used where a counting sort with global atomic counters would otherwise
// serialise on the memory-side atomics: ordering neighbourhood edges by
// column (the transpose) and events by pixel (the per-pixel lists).
#include "common.hpp"

namespace sbc {
namespace {

constexpr int kSortThreads = 256;
constexpr int kSortWaves = kSortThreads / 64;
constexpr int kMaxDigitBits = 8;
constexpr int kMaxRounds = 16;   // 64-item rounds per wave; blocks hold 256 * rounds items

__device__ __forceinline__ int64_t item_count(const int64_t *n_dev, int64_t n_bound) {
    const int64_t n = n_dev ? *n_dev : n_bound;
    return n < 0 ? 0 : (n < n_bound ? n : n_bound);
}

// Lanes of the wave whose digit equals this lane's (among the valid ones).
__device__ __forceinline__ uint64_t same_digit_lanes(int dig, bool valid, int bits) {
    uint64_t match = __ballot(valid);
    for (int bit = 0; bit < bits; ++bit) {
        const int b = (dig >> bit) & 1;
        const uint64_t ones = __ballot(b);
        match &= b ? ones : ~ones;
    }
    return match;
}

// counts[d * n_blocks + b] = items of block b whose digit is d; one LDS add per
// distinct digit of each 64-item round.
template <int R>
__global__ void __launch_bounds__(kSortThreads)
    digit_count_kernel(const int32_t *__restrict__ keys, const int64_t *n_dev, int64_t n_bound,
                       int shift, int bits, int32_t *__restrict__ counts) {
    __shared__ int32_t hist[1 << kMaxDigitBits];
    const int nd = 1 << bits;
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    for (int d = threadIdx.x; d < nd; d += kSortThreads) hist[d] = 0;
    const int64_t n = item_count(n_dev, n_bound);
    const int64_t base = (int64_t)blockIdx.x * (kSortThreads * R) + (int64_t)w * (64 * R);
    int32_t dig[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int64_t i = base + r * 64 + lane;
        dig[r] = i < n ? (keys[i] >> shift) & (nd - 1) : 0;
    }
    __syncthreads();
    const uint64_t lanes_below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const bool valid = base + r * 64 + lane < n;
        const uint64_t match = same_digit_lanes(dig[r], valid, bits);
        if (valid && (match & lanes_below) == 0) atomicAdd(&hist[dig[r]], __popcll(match));
    }
    __syncthreads();
    for (int d = threadIdx.x; d < nd; d += kSortThreads)
        counts[(int64_t)d * gridDim.x + blockIdx.x] = hist[d];
}

// Scatter of block b's items to offsets[d * n_blocks + b] + (rank among the
// block's items with digit d).  The block first orders its items by digit in
// LDS (stable), then writes them out in that order, so each digit's run goes
// to consecutive addresses.  vals_in == nullptr: the value is the item's
// index.
template <int R>
__global__ void __launch_bounds__(kSortThreads)
    digit_scatter_kernel(const int32_t *__restrict__ keys_in, const int32_t *__restrict__ vals_in,
                         const int64_t *n_dev, int64_t n_bound, int shift, int bits,
                         const int32_t *__restrict__ offsets, int32_t *__restrict__ keys_out,
                         int32_t *__restrict__ vals_out) {
    constexpr int CH = kSortThreads * R;
    constexpr int ND = 1 << kMaxDigitBits;
    __shared__ int32_t wcnt[kSortWaves][ND];
    __shared__ int32_t dstart[ND + 1];
    __shared__ int32_t sk[CH];
    __shared__ int32_t sv[CH];
    __shared__ int32_t dbase[ND];  // this block's first output position per digit
    const int nd = 1 << bits;
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    for (int q = threadIdx.x; q < kSortWaves * ND; q += kSortThreads) wcnt[q / ND][q % ND] = 0;
    if (threadIdx.x < nd) dbase[threadIdx.x] = offsets[(int64_t)threadIdx.x * gridDim.x + blockIdx.x];
    const int64_t n = item_count(n_dev, n_bound);
    const int64_t block0 = (int64_t)blockIdx.x * CH;
    const int64_t base = block0 + (int64_t)w * (64 * R);
    int32_t key[R], val[R], dig[R], pos[R];
    // every item of the wave is loaded before the ranking starts
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int64_t i = base + r * 64 + lane;
        const bool valid = i < n;
        key[r] = valid ? keys_in[i] : 0;
        val[r] = valid ? (vals_in ? vals_in[i] : (int32_t)i) : 0;
    }
    __syncthreads();
    const uint64_t lanes_below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const bool valid = base + r * 64 + lane < n;
        dig[r] = (key[r] >> shift) & (nd - 1);
        const uint64_t match = same_digit_lanes(dig[r], valid, bits);
        const int rank = __popcll(match & lanes_below);
        const int before = wcnt[w][dig[r]];   // every lane reads before the leader adds
        pos[r] = before + rank;
        if (valid && rank == 0) wcnt[w][dig[r]] = before + __popcll(match);
    }
    __syncthreads();
    // per digit (one per thread): prefix over the block's waves, and the
    // digit's total; then the block-wide exclusive scan of the totals
    static_assert(ND == kSortThreads, "one digit per thread");
    {
        const int d = threadIdx.x;
        int32_t tot = 0;
#pragma unroll
        for (int q = 0; q < kSortWaves; ++q) {
            const int32_t c = wcnt[q][d];
            wcnt[q][d] = tot;
            tot += c;
        }
        dstart[d] = tot;
    }
    __syncthreads();
    for (int o = 1; o < ND; o <<= 1) {  // inclusive Hillis-Steele scan
        const int32_t add = threadIdx.x >= o ? dstart[threadIdx.x - o] : 0;
        __syncthreads();
        dstart[threadIdx.x] += add;
        __syncthreads();
    }
    {
        const int32_t incl = dstart[threadIdx.x];
        __syncthreads();
        dstart[threadIdx.x + 1] = incl;
        if (threadIdx.x == 0) dstart[0] = 0;
    }
    __syncthreads();
    // the block's items in digit order, in LDS
#pragma unroll
    for (int r = 0; r < R; ++r) {
        if (base + r * 64 + lane < n) {
            const int lp = dstart[dig[r]] + wcnt[w][dig[r]] + pos[r];
            sk[lp] = key[r];
            sv[lp] = val[r];
        }
    }
    __syncthreads();
    const int64_t left = n - block0;
    const int cnt = left < CH ? (int)(left > 0 ? left : 0) : CH;
    for (int t = threadIdx.x; t < cnt; t += kSortThreads) {
        const int32_t k = sk[t];
        const int d = (k >> shift) & (nd - 1);
        const int64_t p = (int64_t)dbase[d] + (t - dstart[d]);
        keys_out[p] = k;
        vals_out[p] = sv[t];
    }
}

// Rounds per wave: small arrays take more, smaller blocks, to fill the device.
int sort_rounds(int64_t n_bound) {
    return n_bound >= ((int64_t)1 << 22) ? 16 : (n_bound >= ((int64_t)1 << 20) ? 8 : 4);
}

// ptr[k] = first position p of the sorted keys with key[p] >= k, k in [0, key_bound]
// (keys in [0, key_bound]).
__global__ void segment_bounds_kernel(const int32_t *__restrict__ sorted, const int64_t *n_dev,
                                      int64_t n_bound, int32_t key_bound,
                                      int32_t *__restrict__ ptr) {
    const int64_t n = item_count(n_dev, n_bound);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (n == 0) {
        for (int64_t k = tid; k <= key_bound; k += stride) ptr[k] = 0;
        return;
    }
    // every k up to the last key is the first key of exactly one item's gap
    for (int64_t p = tid; p < n; p += stride) {
        const int32_t k = sorted[p];
        const int32_t kp = p > 0 ? sorted[p - 1] : -1;
        for (int32_t c = kp + 1; c <= k && c <= key_bound; ++c) ptr[c] = (int32_t)p;
    }
    const int32_t last = sorted[n - 1];
    for (int64_t k = tid; k <= key_bound; k += stride)
        if (k > last) ptr[k] = (int32_t)n;
}

int digit_bits_total(int32_t key_bound) {
    int bits = 1;
    while (bits < 31 && ((int64_t)1 << bits) < (int64_t)key_bound) ++bits;
    return bits;
}


struct SortWs {
    int32_t *ka, *kb, *va, *vb, *counts, *offsets;
    int64_t *total;
    void *scan_ws;
};

SortWs carve_sort(void *base, int64_t n_bound, size_t *bytes) {
    const int64_t n = n_bound > 0 ? n_bound : 1;
    const int64_t chunk = (int64_t)kSortThreads * sort_rounds(n_bound);
    const int64_t nc = ((n + chunk - 1) / chunk) << kMaxDigitBits;
    Carver cv(base);
    SortWs w;
    w.ka = cv.take<int32_t>(n);
    w.kb = cv.take<int32_t>(n);
    w.va = cv.take<int32_t>(n);
    w.vb = cv.take<int32_t>(n);
    w.counts = cv.take<int32_t>(nc);
    w.offsets = cv.take<int32_t>(nc);
    w.total = cv.take<int64_t>(1);
    w.scan_ws = cv.take<char>(scan_workspace_bytes(nc));
    if (bytes) *bytes = cv.used;
    return w;
}

template <int R>
void launch_pass(int64_t nb, const int32_t *kin, const int32_t *vin, const int64_t *n_dev,
                 int64_t n_bound, int shift, int w, int32_t *counts, int32_t *offsets,
                 int32_t *kout, int32_t *vout, bool count, hipStream_t stream) {
    if (count)
        hipLaunchKernelGGL(digit_count_kernel<R>, dim3((unsigned)nb), dim3(kSortThreads), 0,
                           stream, kin, n_dev, n_bound, shift, w, counts);
    else
        hipLaunchKernelGGL(digit_scatter_kernel<R>, dim3((unsigned)nb), dim3(kSortThreads), 0,
                           stream, kin, vin, n_dev, n_bound, shift, w, offsets, kout, vout);
}

}  // namespace

size_t radix_sort_workspace_bytes(int64_t n_bound) {
    size_t bytes = 0;
    carve_sort(nullptr, n_bound, &bytes);
    return bytes;
}

sbc_status radix_sort_pairs(const int32_t *keys, const int32_t *vals, const int64_t *n_dev,
                            int64_t n_bound, int32_t key_bound, int32_t *keys_out,
                            int32_t *vals_out, void *ws, hipStream_t stream) {
    if (n_bound <= 0) return SBC_OK;
    const int R = sort_rounds(n_bound);
    const int64_t nb = (n_bound + (int64_t)kSortThreads * R - 1) / ((int64_t)kSortThreads * R);
    const SortWs sw = carve_sort(ws, n_bound, nullptr);
    const int bits = digit_bits_total(key_bound);
    const int passes = (bits + kMaxDigitBits - 1) / kMaxDigitBits;
    const int width = (bits + passes - 1) / passes;
    const int32_t *kin = keys;
    const int32_t *vin = vals;
    for (int p = 0; p < passes; ++p) {
        const int shift = p * width;
        const int w = bits - shift < width ? bits - shift : width;
        const bool last = p == passes - 1;
        int32_t *kout = last ? keys_out : (p % 2 == 0 ? sw.ka : sw.kb);
        int32_t *vout = last ? vals_out : (p % 2 == 0 ? sw.va : sw.vb);
        const int64_t ncp = nb << w;
        for (int step = 0; step < 2; ++step) {
            const bool count = step == 0;
            switch (R) {
                case 16: launch_pass<16>(nb, kin, vin, n_dev, n_bound, shift, w, sw.counts, sw.offsets, kout, vout, count, stream); break;
                case 8: launch_pass<8>(nb, kin, vin, n_dev, n_bound, shift, w, sw.counts, sw.offsets, kout, vout, count, stream); break;
                default: launch_pass<4>(nb, kin, vin, n_dev, n_bound, shift, w, sw.counts, sw.offsets, kout, vout, count, stream); break;
            }
            SBC_LAUNCH_CHECK();
            if (count) SBC_TRY(exclusive_scan_i32(sw.counts, sw.offsets, ncp, sw.total, sw.scan_ws, stream));
        }
        kin = kout;
        vin = vout;
    }
    return SBC_OK;
}

sbc_status segment_bounds(const int32_t *sorted, const int64_t *n_dev, int64_t n_bound,
                          int32_t key_bound, int32_t *ptr, hipStream_t stream) {
    int64_t blocks = ((n_bound > key_bound ? n_bound : (int64_t)key_bound + 1) + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(segment_bounds_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, sorted,
                       n_dev, n_bound, key_bound, ptr);
    SBC_LAUNCH_CHECK();
    return SBC_OK;
}

}  // namespace sbc
