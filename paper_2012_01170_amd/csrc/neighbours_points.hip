// Ball (optionally k-capped) neighbourhoods of a ragged batch of point clouds
// (Section 3.1, "Neighborhoods"; "Ragged Batching").
//
// Pipeline (all on the caller's stream):
//   1. cell key of every input point: hash(cloud, floor(x / h)) with cell
//      edge h = r (1 + 2^-10) evaluated in float64, so that any pair with
//      float32 d2 < r*r lies in the same or an adjacent cell;
//   2. counting sort of the inputs by key (count, scan, scatter) into a
//      cell table of packed (x, y, z, j) records;
//   3. count pass, one wave per output row: the 27 adjacent cells are hashed,
//      duplicate buckets dropped, candidates tested by the canonical float32
//      distance; row length = min(in-ball count, k_cap);
//   4. scan of the row lengths -> row_ptr (E is read back only on request);
//   5. fill pass, one wave per row: in-ball (d2, j) pairs are staged in LDS,
//      truncated to the k_cap smallest by rank on (d2, j), and written in
//      ascending j by rank on j.  Rows longer than the LDS stage rank against
//      the candidate cells directly (same result, slower).
// A capped search (1 <= k_cap <= kStage) instead runs the fill pass once,
// before the scan, into rows of stride k_cap in the workspace (it also
// writes the row lengths), and copies the rows into place after the scan, so
// the candidates are visited once rather than twice.
// The hash only prunes: buckets shared by distinct cells or clouds add
// candidates that the exact distance and cloud-range tests reject.
#include <cfloat>
#include <climits>

#include "common.hpp"

namespace sbc {
namespace {

constexpr int kWaves = 4;              // waves per block
constexpr int kStage = 512;            // in-ball candidates staged per wave in LDS
constexpr double kCellMargin = 1.0 + 1.0 / 1024.0;

struct PointRec {
    float x, y, z;
    int32_t j;
};

// Make this wave's LDS writes visible to all of its lanes before later reads.
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
    __builtin_amdgcn_wave_barrier();
}

__device__ __forceinline__ uint32_t hash_cell(int32_t b, int32_t cx, int32_t cy, int32_t cz) {
    uint32_t h = (uint32_t)b * 0x9E3779B1u;
    h ^= (uint32_t)cx * 0x85EBCA77u + 0x165667B1u + (h << 6) + (h >> 2);
    h ^= (uint32_t)cy * 0xC2B2AE3Du + 0x27D4EB2Fu + (h << 6) + (h >> 2);
    h ^= (uint32_t)cz * 0x61C88647u + 0x9E3779B9u + (h << 6) + (h >> 2);
    h ^= h >> 15;
    h *= 0x2C1B3C6Du;
    h ^= h >> 12;
    return h;
}

// Bucket of cell (cx, cy, cz) of cloud b, whose inputs are j_lo ..
// j_lo + n_b - 1: every cloud owns the 2 n_b + 1 buckets from 2 j_lo + b, so
// clouds never share a bucket and a cloud's table can be built on its own.
// The result is clamped below T (only malformed splits need it).
__device__ __forceinline__ uint32_t cloud_bucket(int32_t b, int32_t j_lo, int32_t n_b,
                                                 uint32_t T, int32_t cx, int32_t cy, int32_t cz) {
    const uint32_t nb = n_b > 0 ? (uint32_t)n_b : 0u;
    const uint32_t k = 2u * (uint32_t)j_lo + (uint32_t)b + hash_cell(b, cx, cy, cz) % (2u * nb + 1u);
    return k < T ? k : T - 1u;
}

__device__ __forceinline__ int32_t cell_coord(float x, double inv_h) {
    double c = floor((double)x * inv_h);
    // clamping is monotone, so adjacent cells stay adjacent; NaN -> 0
    if (!(c == c)) return 0;
    if (c > 1073741824.0) c = 1073741824.0;
    if (c < -1073741824.0) c = -1073741824.0;
    return (int32_t)c;
}

// index b with splits[b] <= i < splits[b+1] (splits non-decreasing, n_batch+1 long)
__device__ __forceinline__ int32_t cloud_of(const int32_t *splits, int32_t n_batch, int32_t i) {
    int32_t lo = 0, hi = n_batch;  // answer in [0, n_batch)
    while (hi - lo > 1) {
        int32_t mid = (lo + hi) >> 1;
        if (splits[mid] <= i) lo = mid; else hi = mid;
    }
    return lo;
}

// The L lanes of a wave that serve one row (L = 64 or 32): sl is the lane
// within the segment; ballots are restricted to the segment's lanes.
template <int L>
struct Seg {
    int lane, sl, grp;
    uint64_t full;
    __device__ Seg() {
        lane = threadIdx.x & 63;
        sl = lane % L;
        grp = lane / L;
        full = L == 64 ? ~0ull : (((1ull << L) - 1ull) << (grp * L));
    }
    __device__ uint64_t ballot(bool p) const { return __ballot(p) & full; }
    // lanes of the segment below this one among those set in m
    __device__ int below(uint64_t m) const { return __popcll(m & ((1ull << lane) - 1ull)); }
    __device__ int32_t shfl(int32_t v, int q) const { return __shfl(v, grp * L + q, 64); }
};

// Cloud b of the output index i, the same on every lane of the segment, and
// the input range [*j_lo, *j_hi) of that cloud.  The splits are read across
// the segment, L at a time, and b counts the interior splits at or below i,
// which for non-decreasing splits is the bisection's answer.  With fewer
// than L clouds the input splits are read in the same round trip and picked
// out by lane.
template <int L>
__device__ __forceinline__ int32_t seg_cloud(const Seg<L> &sg, const int32_t *__restrict__ out_splits,
                                             const int32_t *__restrict__ in_splits,
                                             int32_t n_batch, int32_t i, int32_t *j_lo,
                                             int32_t *j_hi) {
    const int sl = sg.sl;
    if (n_batch < L) {
        const int32_t so = sl <= n_batch ? out_splits[sl] : 0;
        const int32_t si = sl <= n_batch ? in_splits[sl] : 0;
        const int32_t b = __popcll(sg.ballot(sl >= 1 && sl < n_batch && so <= i));
        *j_lo = sg.shfl(si, b);
        *j_hi = sg.shfl(si, b + 1);
        return b;
    }
    int32_t b = 0;
    for (int32_t base = 1; base < n_batch; base += L) {
        const int32_t k = base + sl;
        b += __popcll(sg.ballot(k < n_batch && out_splits[k] <= i));
    }
    *j_lo = in_splits[b];
    *j_hi = in_splits[b + 1];
    return b;
}

// Canonical float32 squared distance: fixed association and no contraction
// (the rounding intrinsics alone do not stop the compiler from fusing the
// products into the sums; the pragma does).
__device__ __forceinline__ float sq_dist(float ax, float ay, float az, float bx, float by,
                                         float bz) {
#pragma clang fp contract(off)
    const float dx = ax - bx, dy = ay - by, dz = az - bz;
    return (dx * dx + dy * dy) + dz * dz;
}

// Zeroes the cell counts and the status word.
__global__ void init_kernel(int32_t *__restrict__ cell_count, uint32_t table_size,
                            uint32_t *status) {
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    for (int64_t x = gid; x < table_size; x += (int64_t)gridDim.x * blockDim.x) cell_count[x] = 0;
    if (gid == 0) *status = 0u;
}

// Cell key of every input point (and, in the first n_batch + 1 threads, the
// check that the splits run from 0 to n_in / n_out without decreasing).
constexpr int kKeyThreads = 256;
constexpr int kSplitsInLds = 1024;     // key pass: splits bisected in LDS up to this many

__global__ void __launch_bounds__(kKeyThreads)
    key_kernel(const float *__restrict__ x_in, int32_t n_in,
               const int32_t *__restrict__ in_splits, const int32_t *__restrict__ out_splits,
               int32_t n_out, int32_t n_batch, double inv_h, uint32_t T,
               uint32_t *__restrict__ keys, int32_t *__restrict__ counts, uint32_t *status) {
    __shared__ int32_t s_splits[kSplitsInLds];
    const bool lds = n_batch < kSplitsInLds;
    if (lds)
        for (int k = threadIdx.x; k <= n_batch; k += kKeyThreads) s_splits[k] = in_splits[k];
    __syncthreads();
    int32_t j = blockIdx.x * blockDim.x + threadIdx.x;
    if (j <= n_batch) {
        const int32_t b = j;
        bool bad = false;
        if (b == 0) bad = in_splits[0] != 0 || out_splits[0] != 0;
        if (b == n_batch) bad = bad || in_splits[b] != n_in || out_splits[b] != n_out;
        if (b > 0)
            bad = bad || in_splits[b] < in_splits[b - 1] || out_splits[b] < out_splits[b - 1];
        if (bad) atomicOr(status, (uint32_t)kFlagBadSplits);
    }
    if (j >= n_in) return;
    const int32_t *sp = lds ? s_splits : in_splits;
    int32_t b = cloud_of(sp, n_batch, j);
    float x = x_in[3 * (int64_t)j], y = x_in[3 * (int64_t)j + 1], z = x_in[3 * (int64_t)j + 2];
    uint32_t key = cloud_bucket(b, sp[b], sp[b + 1] - sp[b], T, cell_coord(x, inv_h),
                                cell_coord(y, inv_h), cell_coord(z, inv_h));
    keys[j] = key;
    atomicAdd(&counts[key], 1);
}

__global__ void scatter_kernel(const float *__restrict__ x_in, int32_t n_in,
                               const uint32_t *__restrict__ keys, int32_t *__restrict__ cursor,
                               PointRec *__restrict__ table) {
    int32_t j = blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= n_in) return;
    int32_t pos = atomicAdd(&cursor[keys[j]], 1);
    PointRec r;
    r.x = x_in[3 * (int64_t)j];
    r.y = x_in[3 * (int64_t)j + 1];
    r.z = x_in[3 * (int64_t)j + 2];
    r.j = j;
    table[pos] = r;
}

// One workgroup per cloud builds that cloud's cell table (the count, scan
// and scatter of the multi-kernel build, in one launch): counts in LDS when
// the cloud's buckets fit (kLdsBuckets), else in the global count array; the
// scan of the counts runs over the cloud's buckets in chunks with a carried
// total.  Workgroup 0 also clears the status word and checks the splits.
constexpr int kCloudThreads = 512;
constexpr int kLdsBuckets = 8193;      // 2 * 4096 + 1
constexpr int kLdsPoints = 4096;

__global__ void __launch_bounds__(kCloudThreads)
    cloud_table_kernel(const float *__restrict__ x_in, int32_t n_in,
                       const int32_t *__restrict__ in_splits,
                       const int32_t *__restrict__ out_splits, int32_t n_out, int32_t n_batch,
                       double inv_h, uint32_t T, uint32_t *__restrict__ keys,
                       int32_t *__restrict__ counts, int32_t *__restrict__ cell_start,
                       int32_t *__restrict__ cursor, PointRec *__restrict__ table,
                       uint32_t *status) {
    __shared__ int32_t s_cnt[kLdsBuckets];
    __shared__ uint32_t s_key[kLdsPoints];
    __shared__ int32_t wsum[kCloudThreads / 64];
    __shared__ int32_t s_carry;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int b = blockIdx.x;
    if (b == 0) {
        if (tid == 0) *status = 0u;
        __syncthreads();
        for (int32_t k = tid; k <= n_batch; k += kCloudThreads) {
            bool bad = false;
            if (k == 0) bad = in_splits[0] != 0 || out_splits[0] != 0;
            if (k == n_batch) bad = bad || in_splits[k] != n_in || out_splits[k] != n_out;
            if (k > 0) bad = bad || in_splits[k] < in_splits[k - 1] || out_splits[k] < out_splits[k - 1];
            if (bad) atomicOr(status, (uint32_t)kFlagBadSplits);
        }
    }
    const int32_t j_lo = min(max(in_splits[b], 0), n_in);
    const int32_t j_hi = min(max(in_splits[b + 1], j_lo), n_in);
    const int32_t n_b = j_hi - j_lo;
    const uint32_t off = 2u * (uint32_t)j_lo + (uint32_t)b;
    const uint32_t Tb = 2u * (uint32_t)n_b + 1u;
    if (off >= T) return;  // only malformed splits get here (the whole workgroup)
    const uint32_t nbk = off + Tb <= T ? Tb : T - off;  // buckets written
    const bool lds = Tb <= (uint32_t)kLdsBuckets;
    int32_t *cnt = lds ? s_cnt : counts + off;
    for (uint32_t k = tid; k < nbk; k += kCloudThreads) cnt[k] = 0;
    __syncthreads();
    for (int32_t p = tid; p < n_b; p += kCloudThreads) {
        const int32_t j = j_lo + p;
        const uint32_t key = cloud_bucket(b, j_lo, n_b, T, cell_coord(x_in[3 * (int64_t)j], inv_h),
                                          cell_coord(x_in[3 * (int64_t)j + 1], inv_h),
                                          cell_coord(x_in[3 * (int64_t)j + 2], inv_h)) - off;
        if (lds) s_key[p] = key; else keys[j] = key;
        atomicAdd(&cnt[key], 1);
    }
    __syncthreads();
    // exclusive scan of the cloud's counts, in place, chunk by chunk
    if (tid == 0) s_carry = 0;
    __syncthreads();
    for (uint32_t c0 = 0; c0 < nbk; c0 += 4 * kCloudThreads) {
        int32_t v[4], sum = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const uint32_t k = c0 + 4 * tid + q;
            v[q] = k < nbk ? cnt[k] : 0;
            sum += v[q];
        }
        int32_t x = sum;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int32_t y = __shfl_up(x, d, 64);
            if (lane >= d) x += y;
        }
        if (lane == 63) wsum[wave] = x;
        __syncthreads();
        int32_t before = s_carry, tot = 0;
#pragma unroll
        for (int w = 0; w < kCloudThreads / 64; ++w) {
            before += w < wave ? wsum[w] : 0;
            tot += wsum[w];
        }
        int32_t run = before + x - sum;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const uint32_t k = c0 + 4 * tid + q;
            if (k < nbk) {
                cnt[k] = run;  // now the bucket's start within the cloud
                cell_start[off + k] = j_lo + run;
                if (!lds) cursor[off + k] = run;
            }
            run += v[q];
        }
        __syncthreads();
        if (tid == 0) s_carry += tot;
        __syncthreads();
    }
    if (tid == 0) cell_start[off + nbk] = j_lo + n_b;  // the next cloud's start, or the end
    __syncthreads();
    // scatter the records; the bucket starts serve as cursors
    int32_t *cur = lds ? s_cnt : cursor + off;
    for (int32_t p = tid; p < n_b; p += kCloudThreads) {
        const int32_t j = j_lo + p;
        const uint32_t key = lds ? s_key[p] : keys[j];
        const int32_t pos = atomicAdd(&cur[key], 1);
        PointRec r;
        r.x = x_in[3 * (int64_t)j];
        r.y = x_in[3 * (int64_t)j + 1];
        r.z = x_in[3 * (int64_t)j + 2];
        r.j = j;
        table[j_lo + pos] = r;
    }
}

struct RowCtx {
    float qx, qy, qz;
    int32_t j_lo, j_hi;  // input range of the row's cloud
    float r2;
};

// Per segment: bucket ranges of the 27 cells around the query, duplicates
// removed; lane k < 27 of the segment holds cell k.  Returns the candidate
// count; lane k's range start and its exclusive offset into the flattened
// candidate list go to lds_start/lds_off (27 entries each).
template <int L>
__device__ int32_t gather_buckets(const Seg<L> &sg, const RowCtx &c, int32_t b, double inv_h,
                                  uint32_t T, const int32_t *__restrict__ cell_start,
                                  int32_t *lds_start, int32_t *lds_off) {
    static_assert(L >= 27, "a lane per cell");
    const int sl = sg.sl;
    int32_t cx = cell_coord(c.qx, inv_h), cy = cell_coord(c.qy, inv_h), cz = cell_coord(c.qz, inv_h);
    uint32_t bucket = 0xFFFFFFFFu;
    int32_t s = 0, len = 0;
    if (sl < 27) {
        int32_t dx = sl % 3 - 1, dy = (sl / 3) % 3 - 1, dz = sl / 9 - 1;
        bucket = cloud_bucket(b, c.j_lo, c.j_hi - c.j_lo, T, cx + dx, cy + dy, cz + dz);
    }
    bool dup = false;
    for (int q = 0; q < 27; ++q) {
        uint32_t bq = (uint32_t)sg.shfl((int32_t)bucket, q);
        if (q < sl && bq == bucket) dup = true;
    }
    if (sl < 27 && !dup) {
        s = cell_start[bucket];
        len = cell_start[bucket + 1] - s;
    }
    // exclusive scan of len over the segment
    int32_t incl = len;
#pragma unroll
    for (int d = 1; d < L; d <<= 1) {
        int32_t y = __shfl_up(incl, d, 64);
        if (sl >= d) incl += y;
    }
    int32_t total = sg.shfl(incl, L - 1);
    if (sl < 27) {
        lds_start[sl] = s;
        lds_off[sl] = incl - len;
    }
    return total;
}

// Candidate c (0 <= c < total) of the flattened bucket list -> table position.
__device__ __forceinline__ int32_t candidate_pos(int32_t c, const int32_t *lds_start,
                                                 const int32_t *lds_off) {
    int32_t k = 0;
#pragma unroll
    for (int q = 1; q < 27; ++q) k = (lds_off[q] <= c) ? q : k;
    // several lanes may share an offset when buckets are empty or duplicate:
    // the largest q with off <= c has a non-empty range containing c
    return lds_start[k] + (c - lds_off[k]);
}

__device__ __forceinline__ bool in_ball(const RowCtx &c, const PointRec &p, float *d2) {
    if (p.j < c.j_lo || p.j >= c.j_hi) return false;
    float d = sq_dist(c.qx, c.qy, c.qz, p.x, p.y, p.z);
    *d2 = d;
    return d < c.r2;
}

__device__ __forceinline__ bool key_less(float da, int32_t ja, float db, int32_t jb) {
    return da < db || (da == db && ja < jb);
}

// kMode: 0 count pass; 1 fill pass into the CSR (row i at row_ptr[i]);
// 2 fill pass into rows of stride k_cap (row i at i * k_cap, col_capacity =
// n_out * k_cap), writing the row lengths too.  A row takes L lanes (a wave
// holds 64 / L rows), with a stage of kStage * L / 64 candidates.
template <int kMode, int L>
__global__ void __launch_bounds__(kWaves * 64)
    rows_kernel(const float *__restrict__ x_out, int32_t n_out,
                const int32_t *__restrict__ in_splits, const int32_t *__restrict__ out_splits,
                int32_t n_batch, float radius, int32_t k_cap, double inv_h, uint32_t T,
                const int32_t *__restrict__ cell_start, const PointRec *__restrict__ table,
                int32_t *__restrict__ row_len, const int32_t *__restrict__ row_ptr,
                int32_t *__restrict__ col_idx, int64_t col_capacity) {
    constexpr int G = 64 / L;                 // rows per wave
    constexpr int kStageL = kStage / G;       // staged candidates per row
    constexpr int kRows = kWaves * G;         // rows per block
    __shared__ int32_t s_start[kRows][27];
    __shared__ int32_t s_off[kRows][27];
    constexpr bool kFill = kMode != 0;
    __shared__ float s_d2[kFill ? kRows : 1][kFill ? kStageL : 1];
    __shared__ int32_t s_j[kFill ? kRows : 1][kFill ? kStageL : 1];

    const Seg<L> sg;
    const int sl = sg.sl;
    const int rw = (threadIdx.x >> 6) * G + sg.grp;  // row within the block
    const int32_t i = blockIdx.x * kRows + rw;
    if (i >= n_out) return;  // a segment leaves on its own: no block barrier below

    RowCtx c;
    c.qx = x_out[3 * (int64_t)i];
    c.qy = x_out[3 * (int64_t)i + 1];
    c.qz = x_out[3 * (int64_t)i + 2];
    const int32_t b = seg_cloud(sg, out_splits, in_splits, n_batch, i, &c.j_lo, &c.j_hi);
    c.r2 = __fmul_rn(radius, radius);

    const int32_t total = gather_buckets(sg, c, b, inv_h, T, cell_start, s_start[rw], s_off[rw]);
    wave_lds_sync();

    if (!kFill) {
        int32_t n = 0;
        for (int32_t base = 0; base < total; base += L) {
            int32_t cc = base + sl;
            bool hit = false;
            if (cc < total) {
                PointRec p = table[candidate_pos(cc, s_start[rw], s_off[rw])];
                float d2;
                hit = in_ball(c, p, &d2);
            }
            n += __popcll(sg.ballot(hit));
        }
        if (sl == 0) row_len[i] = (k_cap > 0 && n > k_cap) ? k_cap : n;
        return;
    }

    // ---- fill pass: stage the in-ball candidates
    int32_t n = 0;
    for (int32_t base = 0; base < total; base += L) {
        int32_t cc = base + sl;
        bool hit = false;
        float d2 = 0.f;
        int32_t j = 0;
        if (cc < total) {
            PointRec p = table[candidate_pos(cc, s_start[rw], s_off[rw])];
            hit = in_ball(c, p, &d2);
            j = p.j;
        }
        const uint64_t mask = sg.ballot(hit);
        int32_t slot = n + sg.below(mask);
        if (hit && slot < kStageL) {
            s_d2[rw][slot] = d2;
            s_j[rw][slot] = j;
        }
        n += __popcll(mask);
    }
    wave_lds_sync();
    const int64_t out0 = kMode == 2 ? (int64_t)i * k_cap : (int64_t)row_ptr[i];
    const bool capped = k_cap > 0 && n > k_cap;
    const int32_t n_keep = capped ? k_cap : n;
    if (kMode == 2 && sl == 0) row_len[i] = n_keep;

    if (n <= kStageL) {
        if (capped) {
            // keep the entries whose rank on (d2, j) is below k_cap; a dropped
            // entry gets bit 31 set in its staged j, which orders it (as an
            // unsigned number) after every kept one
            constexpr int kPerLane = kStageL / L;
            bool drop[kPerLane];
#pragma unroll
            for (int u = 0; u < kPerLane; ++u) {
                const int32_t a = sl + L * u;
                drop[u] = false;
                if (a < n) {
                    const float da = s_d2[rw][a];
                    const int32_t ja = s_j[rw][a];
                    int32_t rank = 0;
                    for (int32_t q = 0; q < n; ++q) rank += key_less(s_d2[rw][q], s_j[rw][q], da, ja);
                    drop[u] = rank >= k_cap;
                }
            }
            wave_lds_sync();
#pragma unroll
            for (int u = 0; u < kPerLane; ++u)
                if (drop[u]) s_j[rw][sl + L * u] |= INT32_MIN;
            wave_lds_sync();
        }
        // position among the kept entries by rank on j
        for (int32_t a = sl; a < n; a += L) {
            const uint32_t ja = (uint32_t)s_j[rw][a];
            if (ja & 0x80000000u) continue;
            int32_t pos = 0;
            for (int32_t q = 0; q < n; ++q) pos += ((uint32_t)s_j[rw][q] < ja) ? 1 : 0;
            int64_t dst = (int64_t)out0 + pos;
            if (dst < col_capacity) col_idx[dst] = (int32_t)ja;
        }
        return;
    }

    // ---- long rows (more in-ball candidates than the LDS stage holds).
    // Keys (d2, j) are distinct; order them as the 64-bit integer
    // (bits(d2) << 32) | j (d2 >= 0, so its bit pattern orders like its value).
    uint64_t threshold = ~0ull;  // keep every in-ball key <= threshold
    if (capped) {
        // smallest K with #{key <= K} >= k_cap, by bisection on K
        uint64_t lo = 0, hi = ~0ull;
        while (lo < hi) {
            const uint64_t mid = lo + ((hi - lo) >> 1);
            int32_t cnt = 0;
            for (int32_t base = 0; base < total; base += L) {
                int32_t cc = base + sl;
                bool le = false;
                if (cc < total) {
                    PointRec p = table[candidate_pos(cc, s_start[rw], s_off[rw])];
                    float d2;
                    if (in_ball(c, p, &d2))
                        le = (((uint64_t)__float_as_uint(d2) << 32) | (uint32_t)p.j) <= mid;
                }
                cnt += __popcll(sg.ballot(le));
            }
            if (cnt >= k_cap) hi = mid; else lo = mid + 1;
        }
        threshold = lo;
    }
    // stage the kept column indices when they fit, else rank against the cells
    const bool staged = n_keep <= kStageL;
    int32_t m = 0;
    for (int32_t base = 0; base < total; base += L) {
        int32_t cc = base + sl;
        bool keep = false;
        int32_t j = 0;
        if (cc < total) {
            PointRec p = table[candidate_pos(cc, s_start[rw], s_off[rw])];
            float d2;
            if (in_ball(c, p, &d2)) {
                keep = (((uint64_t)__float_as_uint(d2) << 32) | (uint32_t)p.j) <= threshold;
                j = p.j;
            }
        }
        const uint64_t mask = sg.ballot(keep);
        if (staged) {
            int32_t slot = m + sg.below(mask);
            if (keep) s_j[rw][slot] = j;
        } else if (keep) {
            int32_t pos = 0;
            for (int32_t q = 0; q < total; ++q) {
                PointRec o = table[candidate_pos(q, s_start[rw], s_off[rw])];
                float db;
                if (in_ball(c, o, &db) && o.j < j &&
                    (((uint64_t)__float_as_uint(db) << 32) | (uint32_t)o.j) <= threshold)
                    ++pos;
            }
            int64_t dst = (int64_t)out0 + pos;
            if (dst < col_capacity) col_idx[dst] = j;
        }
        m += __popcll(mask);
    }
    if (staged) {
        wave_lds_sync();
        for (int32_t a = sl; a < m; a += L) {
            int32_t ja = s_j[rw][a];
            int32_t pos = 0;
            for (int32_t q = 0; q < m; ++q) pos += (s_j[rw][q] < ja) ? 1 : 0;
            int64_t dst = (int64_t)out0 + pos;
            if (dst < col_capacity) col_idx[dst] = ja;
        }
    }
}

// col_idx[row_ptr[i] + s] = rows[i * k_cap + s] for s < row_len[i]
__global__ void compact_rows_kernel(const int32_t *__restrict__ rows,
                                    const int32_t *__restrict__ row_len,
                                    const int32_t *__restrict__ row_ptr, int32_t n_out,
                                    int32_t k_cap, int32_t *__restrict__ col_idx,
                                    int64_t col_capacity) {
    const int64_t total = (int64_t)n_out * k_cap;
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < total;
         q += (int64_t)gridDim.x * blockDim.x) {
        const int32_t i = (int32_t)(q / k_cap), sl = (int32_t)(q % k_cap);
        if (sl < row_len[i]) {
            const int64_t dst = (int64_t)row_ptr[i] + sl;
            if (dst < col_capacity) col_idx[dst] = rows[q];
        }
    }
}

bool one_pass(int32_t k_cap) { return k_cap >= 1 && k_cap <= kStage; }

// Two rows per wave when there are at least twice as many rows as the waves
// the chip holds at once (eight per SIMD, four SIMDs per CU); fewer rows keep
// a wave each, so that they still spread over the whole chip.
bool pair_rows(int32_t n_out) { return (int64_t)n_out >= 64LL * device_cus(); }

// rows_kernel<kMode, 32 or 64 lanes per row> over n_out (the second argument)
template <int kMode, typename... Args>
void launch_rows(bool pair, hipStream_t stream, const float *x_out, int32_t n_out,
                 Args... args) {
    const dim3 block(kWaves * 64);
    if (pair)
        hipLaunchKernelGGL((rows_kernel<kMode, 32>), dim3(grid_for(n_out, 2 * kWaves)), block, 0,
                           stream, x_out, n_out, args...);
    else
        hipLaunchKernelGGL((rows_kernel<kMode, 64>), dim3(grid_for(n_out, kWaves)), block, 0,
                           stream, x_out, n_out, args...);
}

// Buckets of all clouds: 2 n_b + 1 per cloud.
uint32_t table_size_for(int32_t n_in, int32_t n_batch) {
    return 2u * (uint32_t)(n_in > 0 ? n_in : 0) + (uint32_t)(n_batch > 0 ? n_batch : 1);
}

struct PointsWs {
    uint32_t *keys;
    int32_t *cell_count;
    int32_t *cell_start;
    int32_t *cursor;
    PointRec *table;
    int32_t *row_len;
    int32_t *rows;  // capped one-pass search: n_out rows of stride k_cap
    int64_t *total;
    uint32_t *status;
    void *scan_ws;
};

PointsWs carve_points(void *base, int32_t n_in, int32_t n_out, int32_t n_batch,
                      int32_t k_cap, size_t *bytes) {
    Carver cv(base);
    const uint32_t T = table_size_for(n_in, n_batch);
    PointsWs w;
    w.keys = cv.take<uint32_t>(n_in);
    w.cell_count = cv.take<int32_t>(T);
    w.cell_start = cv.take<int32_t>((size_t)T + 1);
    w.cursor = cv.take<int32_t>((size_t)T + 1);
    w.table = cv.take<PointRec>(n_in);
    w.row_len = cv.take<int32_t>(n_out);
    w.rows = cv.take<int32_t>(one_pass(k_cap) ? (size_t)n_out * k_cap : 0);
    w.total = cv.take<int64_t>(2);
    w.status = cv.take<uint32_t>(4);
    int64_t m = (int64_t)T > (int64_t)n_out ? (int64_t)T : (int64_t)n_out;
    w.scan_ws = cv.take<char>(scan_workspace_bytes(m));
    if (bytes) *bytes = cv.used;
    return w;
}

}  // namespace
}  // namespace sbc

using namespace sbc;

extern "C" size_t sbc_points_workspace_size(int32_t n_in, int32_t n_out, int32_t n_batch,
                                            int32_t k_cap) {
    size_t bytes = 0;
    carve_points(nullptr, n_in < 0 ? 0 : n_in, n_out < 0 ? 0 : n_out, n_batch, k_cap, &bytes);
    return bytes;
}

extern "C" sbc_status sbc_neighbour_search_points(
    const float *x_in, int32_t n_in, const int32_t *in_splits, const float *x_out, int32_t n_out,
    const int32_t *out_splits, int32_t n_batch, float radius, int32_t k_cap, int32_t *row_ptr,
    int32_t *col_idx, int64_t col_capacity, int64_t *nnz_host, void *workspace,
    size_t workspace_bytes, hipStream_t stream) {
    clear_error();
    if (n_in < 0 || n_out < 0 || n_batch < 1)
        return fail(SBC_ERR_INVALID_ARG, "n_in, n_out must be >= 0 and n_batch >= 1");
    if (!(radius > 0.f) || !(radius < FLT_MAX))
        return fail(SBC_ERR_INVALID_ARG, "radius must be finite and > 0");
    if (!row_ptr || !in_splits || !out_splits || (n_in > 0 && !x_in) || (n_out > 0 && !x_out))
        return fail(SBC_ERR_INVALID_ARG, "null pointer argument");
    if (col_capacity < 0 || (col_capacity > 0 && !col_idx))
        return fail(SBC_ERR_INVALID_ARG, "col_idx is null or col_capacity < 0");
    size_t need = 0;
    PointsWs ws = carve_points(workspace, n_in, n_out, n_batch, k_cap, &need);
    if (!workspace || workspace_bytes < need)
        return fail(SBC_ERR_WORKSPACE, "workspace smaller than sbc_points_workspace_size()");

    if (n_in > (1 << 30)) return fail(SBC_ERR_INVALID_ARG, "n_in must be at most 2^30");
    const uint32_t T = table_size_for(n_in, n_batch);
    const double inv_h = 1.0 / ((double)radius * kCellMargin);

    if ((int64_t)n_in <= 1024 * (int64_t)n_batch) {
        // clouds of about a thousand points or fewer on average: one workgroup
        // per cloud builds its table in one launch
        hipLaunchKernelGGL(cloud_table_kernel, dim3((unsigned)n_batch), dim3(kCloudThreads), 0,
                           stream, x_in, n_in, in_splits, out_splits, n_out, n_batch, inv_h, T,
                           ws.keys, ws.cell_count, ws.cell_start, ws.cursor, ws.table, ws.status);
        SBC_LAUNCH_CHECK();
    } else {
        const int g = grid_for(T, 256) < 1024 ? grid_for(T, 256) : 1024;
        hipLaunchKernelGGL(init_kernel, dim3(g), dim3(256), 0, stream, ws.cell_count, T,
                           ws.status);
        SBC_LAUNCH_CHECK();
        const int64_t kn = (int64_t)n_in > (int64_t)n_batch + 1 ? n_in : (int64_t)n_batch + 1;
        hipLaunchKernelGGL(key_kernel, dim3(grid_for(kn, kKeyThreads)), dim3(kKeyThreads), 0,
                           stream, x_in, n_in,
                           in_splits, out_splits, n_out, n_batch, inv_h, T, ws.keys,
                           ws.cell_count, ws.status);
        SBC_LAUNCH_CHECK();
        SBC_TRY(exclusive_scan_i32(ws.cell_count, ws.cell_start, T, ws.total + 1, ws.scan_ws,
                                   stream, ws.cursor));
        if (n_in > 0) {
            hipLaunchKernelGGL(scatter_kernel, dim3(grid_for(n_in, 256)), dim3(256), 0, stream,
                               x_in, n_in, ws.keys, ws.cursor, ws.table);
            SBC_LAUNCH_CHECK();
        }
    }
    const bool pair = pair_rows(n_out);
    const bool single = one_pass(k_cap);
    if (n_out > 0) {
        trace_before("points_count", stream);
        if (single)
            launch_rows<2>(pair, stream, x_out, n_out, in_splits, out_splits, n_batch, radius, k_cap, inv_h,
                               T, ws.cell_start, ws.table, ws.row_len,
                               (const int32_t *)nullptr, ws.rows, (int64_t)n_out * k_cap);
        else
            launch_rows<0>(pair, stream, x_out, n_out, in_splits, out_splits, n_batch, radius, k_cap, inv_h,
                               T, ws.cell_start, ws.table, ws.row_len,
                               (const int32_t *)nullptr, (int32_t *)nullptr, (int64_t)0);
        SBC_LAUNCH_CHECK();
        trace_after("points_count", stream);
    }
    SBC_TRY(exclusive_scan_i32(ws.row_len, row_ptr, n_out, ws.total, ws.scan_ws, stream));

    if (nnz_host) {
        int64_t host[2];
        uint32_t st = 0;
        SBC_HIP_TRY(hipMemcpyAsync(host, ws.total, sizeof(host), hipMemcpyDeviceToHost, stream));
        SBC_HIP_TRY(hipMemcpyAsync(&st, ws.status, sizeof(st), hipMemcpyDeviceToHost, stream));
        SBC_HIP_TRY(hipStreamSynchronize(stream));
        *nnz_host = host[0];
        if (st & kFlagBadSplits)
            return fail(SBC_ERR_OUT_OF_RANGE,
                        "splits must be non-decreasing from 0 to n_in / n_out");
        if (host[0] > (int64_t)INT32_MAX) return fail(SBC_ERR_OVERFLOW, "2^31 or more edges");
        if (host[0] > col_capacity)
            return fail(SBC_ERR_CAPACITY, "col_capacity " + std::to_string(col_capacity) +
                                              " < E = " + std::to_string(host[0]));
    }
    if (n_out > 0 && col_capacity > 0) {
        trace_before("points_fill", stream);
        if (single) {
            const int64_t total = (int64_t)n_out * k_cap;
            int64_t g = (total + 255) / 256;
            if (g > 8192) g = 8192;
            hipLaunchKernelGGL(compact_rows_kernel, dim3((unsigned)g), dim3(256), 0, stream,
                               ws.rows, ws.row_len, row_ptr, n_out, k_cap, col_idx,
                               col_capacity);
        } else {
            launch_rows<1>(pair, stream, x_out, n_out, in_splits, out_splits, n_batch, radius, k_cap,
                               inv_h, T, ws.cell_start, ws.table, ws.row_len, row_ptr,
                               col_idx, col_capacity);
        }
        SBC_LAUNCH_CHECK();
        trace_after("points_fill", stream);
    }
    return SBC_OK;
}
