// The leaky integrate-and-fire event sampler (the supplementary's event network
// details, and Section 4's stream hierarchy): it turns an event stream into the
// next, coarser one.  Each output cell holds a potential that decays with the
// time since its last update; every input event in its receptive field adds
// 1/n (n = how many cells that event reaches), and when the potential exceeds
// the threshold it is reset and the cell emits an event at the input's time.
//
// A cell's potential depends only on the events of its own receptive field, in
// stream order, so the cells run in parallel:
//   1. each pixel's events are listed, sorted by event index, with their times
//      alongside (counted, placed, then sorted within each pixel; the count
//      also clears the spike flags);
//   2. blocks of 16 cells (8 for kernels of 4 and 5), a wave per cell: the
//      wave stages the lists of its cell's k x k input pixels in LDS and merges
//      them in parallel, each entry finding its place by binary searches in
//      the other lists; the decay factors exp(-(t_s - t_{s-1}) / decay) of the
//      merged sequence do not depend on the potential and are computed in
//      parallel too.  Then one wave runs the block's recursions
//      v = V e_s + 1/n_s (threshold, reset; float64) side by side, a lane per
//      cell; a spike marks its merged entry, and every wave then sets
//      flag[i * slots + slot] for the spikes of its cell (slot: the cell's
//      row-major place among the cells event i reaches).  A cell with more
//      events than the staging holds runs the same recursion on one lane of
//      another wave, merging its lists from global memory;
//   3. a scan over the flags gives every spike its place in the output, which
//      is thereby ordered by input event, then cell row, then cell column (the
//      sequential emission order), and a last kernel writes the events.
#include "common.hpp"
#include "pixel_lists.hpp"

namespace sbc {
namespace {

constexpr int kLifThreads = 64;  // a wave
constexpr int kLifMaxKernel = 5;

struct LifArgs {
    const int32_t *px, *py;
    int32_t n, W, H, Wo, Ho, k, S, pad, nsd;  // nsd: cells per dimension one input can reach
    double decay, thresh, reset;
    const int32_t *pix_start, *list, *list_t;
    int32_t *flags;                           // [n * nsd * nsd]
    uint32_t *status;                         // kFlagInternal on a bad flag index
};

// Marks the spike of event `ev` at its cell slot `slot`.  Both come out of the
// kernel's own merge, so they are always in range; the check keeps a defect
// there from turning into a store outside the flags (it raises the status
// word, which the synchronising call reports, instead).
__device__ __forceinline__ void mark_spike(const LifArgs &A, int64_t ev, int64_t slot) {
    const int64_t nslots = (int64_t)A.nsd * A.nsd;
    if (ev >= 0 && ev < A.n && slot >= 0 && slot < nslots)
        A.flags[ev * nslots + slot] = 1;
    else
        atomicOr(A.status, kFlagInternal);
}

// Cells o (one dimension) whose receptive field [o*S - pad, o*S - pad + k)
// holds input coordinate x: lo..hi (empty when hi < lo).
__device__ __forceinline__ void cell_range(int32_t x, const LifArgs &A, int32_t n_out,
                                           int32_t &lo, int32_t &hi) {
    const int32_t a = x + A.pad - A.k + 1;  // o * S >= a
    lo = a <= 0 ? 0 : (a + A.S - 1) / A.S;
    hi = (x + A.pad) / A.S;
    hi = hi < n_out - 1 ? hi : n_out - 1;
}

// The receptive field of cell (ox, oy): list q (row-major over the k x k
// pixels) starts at *start and holds *len events; inc is 1/n of its pixel and
// slot the cell's place among the cells that pixel reaches.  Off the sensor:
// an empty list.
__device__ __forceinline__ void field_list(const LifArgs &A, int32_t ox, int32_t oy, int q,
                                           int32_t &start, int32_t &len, double &inc,
                                           int32_t &slot) {
    const int32_t x = ox * A.S - A.pad + q % A.k, y = oy * A.S - A.pad + q / A.k;
    start = len = slot = 0;
    inc = 0.0;
    if (x < 0 || x >= A.W || y < 0 || y >= A.H) return;
    const int32_t p = y * A.W + x;
    start = A.pix_start[p];
    len = A.pix_start[p + 1] - start;
    int32_t lx, hx, ly, hy;
    cell_range(x, A, A.Wo, lx, hx);
    cell_range(y, A, A.Ho, ly, hy);
    inc = 1.0 / (double)((hx - lx + 1) * (hy - ly + 1));  // this cell is one of them
    slot = (oy - ly) * A.nsd + (ox - lx);
}

// One cell on one thread: a K*K-way merge of the lists from global memory,
// the earliest head first, advancing the potential at each event.
template <int K>
__device__ void cell_sequential(const LifArgs &A, int32_t ox, int32_t oy) {
#pragma clang fp contract(off)
    constexpr int Q = K * K;
    constexpr int32_t kNone = INT32_MAX;
    int32_t pos[Q], end[Q], head[Q], head_t[Q], slot[Q];
    double inc[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        int32_t len;
        field_list(A, ox, oy, q, pos[q], len, inc[q], slot[q]);
        end[q] = pos[q] + len;
        head[q] = pos[q] < end[q] ? A.list[pos[q]] : kNone;
        head_t[q] = pos[q] < end[q] ? A.list_t[pos[q]] : 0;
    }
    double V = 0.0, T = 0.0;
    for (;;) {
        int32_t best = kNone, bt = 0, bs = 0, bq = -1;
        double binc = 0.0;
#pragma unroll
        for (int q = 0; q < Q; ++q)
            if (head[q] < best) {
                best = head[q];
                bt = head_t[q];
                bs = slot[q];
                binc = inc[q];
                bq = q;
            }
        if (best == kNone) break;
        int32_t np = 0, ne = 0;
#pragma unroll
        for (int q = 0; q < Q; ++q)
            if (q == bq) {
                np = pos[q] + 1;
                ne = end[q];
            }
        const bool more = np < ne;
        const int32_t nh = more ? A.list[np] : kNone;
        const int32_t nt = more ? A.list_t[np] : 0;
#pragma unroll
        for (int q = 0; q < Q; ++q)
            if (q == bq) {
                pos[q] = np;
                head[q] = nh;
                head_t[q] = nt;
            }
        const double ti = (double)bt;
        double v = V * exp(-(ti - T) / A.decay) + binc;
        if (v > A.thresh) {
            v = A.reset;
            mark_spike(A, best, bs);
        }
        V = v;
        T = ti;
    }
}

// Cells per block (a wave each while staging and merging; their recursions
// then run side by side on one wave, a lane per cell), and the LDS sizes.
template <int K>
struct LifTile {
    static constexpr int kCells = K <= 3 ? 16 : 8;
    static constexpr int kStage = 512;                // one cell's events, staged
    static constexpr int kMerged = kCells * 256;      // the block's merged events
};

template <int K>
__global__ void __launch_bounds__(LifTile<K>::kCells * 64) lif_cell_kernel(LifArgs A) {
#pragma clang fp contract(off)
    constexpr int Q = K * K;
    constexpr int C = LifTile<K>::kCells, S = LifTile<K>::kStage, MG = LifTile<K>::kMerged;
    __shared__ int32_t s_idx[C][S];   // each wave's staged lists (list q from off[q])
    __shared__ int32_t s_t[C][S];
    __shared__ int32_t m_idx[MG];     // merged sequences, cell w's from s_moff[w]
    __shared__ int32_t m_t[MG];
    __shared__ uint8_t m_q[MG];
    __shared__ double m_e[MG];        // decay factor of each merged event
    __shared__ int32_t s_start[C][Q], s_len[C][Q], s_slot[C][Q], s_L[C], s_moff[C];
    __shared__ double s_inc[C][Q];
    const int w = threadIdx.x / kLifThreads, lane = threadIdx.x % kLifThreads;
    const int64_t cells = (int64_t)A.Wo * A.Ho;
    const int64_t cell = (int64_t)blockIdx.x * C + w;
    const bool valid = cell < cells;
    const int32_t ox = valid ? (int32_t)(cell % A.Wo) : 0, oy = valid ? (int32_t)(cell / A.Wo) : 0;
    if (valid && lane < Q) {
        int32_t start, len, slot;
        double inc;
        field_list(A, ox, oy, lane, start, len, inc, slot);
        s_start[w][lane] = start;
        s_len[w][lane] = len;
        s_slot[w][lane] = slot;
        s_inc[w][lane] = inc;
    }
    __syncthreads();
    // list offsets (every lane of the wave keeps them) and the longest list
    int32_t off[Q + 1], longest = 0;
    off[0] = 0;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int32_t len = valid ? s_len[w][q] : 0;
        off[q + 1] = off[q] + len;
        longest = len > longest ? len : longest;
    }
    const int32_t L = off[Q];
    if (lane == 0) s_L[w] = L;
    __syncthreads();
    if (threadIdx.x == 0) {  // merged space: cells that fit, in order; the rest run alone
        int32_t o = 0;
        for (int c = 0; c < C; ++c) {
            const bool fits = s_L[c] <= S && o + s_L[c] <= MG;
            s_moff[c] = fits ? o : -1;
            o += fits ? s_L[c] : 0;
        }
    }
    __syncthreads();
    const int32_t mo = s_moff[w];
    const bool staged = valid && mo >= 0;
    if (staged) {
        // stage the lists: the first 64 events of every list in one round of
        // independent loads, longer lists after
        int32_t vi[Q], vt[Q];
#pragma unroll
        for (int q = 0; q < Q; ++q)
            if (lane < off[q + 1] - off[q]) {
                vi[q] = A.list[s_start[w][q] + lane];
                vt[q] = A.list_t[s_start[w][q] + lane];
            }
#pragma unroll
        for (int q = 0; q < Q; ++q)
            if (lane < off[q + 1] - off[q]) {
                s_idx[w][off[q] + lane] = vi[q];
                s_t[w][off[q] + lane] = vt[q];
            }
        if (longest > kLifThreads)
            for (int q = 0; q < Q; ++q)
                for (int32_t j = kLifThreads + lane; j < off[q + 1] - off[q]; j += kLifThreads) {
                    s_idx[w][off[q] + j] = A.list[s_start[w][q] + j];
                    s_t[w][off[q] + j] = A.list_t[s_start[w][q] + j];
                }
    }
    __syncthreads();
    if (staged) {
        // merge: an entry's place is its place in its own list plus, for every
        // other list, the entries there with a smaller event index (binary
        // searches run in lockstep over the lists, so their reads overlap)
        const int steps = 32 - __clz(longest);  // halvings that empty the longest range
        const int32_t *si = s_idx[w];
        for (int32_t e = lane; e < L; e += kLifThreads) {
            int q = 0;
#pragma unroll
            for (int q2 = 1; q2 < Q; ++q2) q += e >= off[q2] ? 1 : 0;
            const int32_t idx = si[e];
            int32_t base[Q], cnt[Q];
#pragma unroll
            for (int q2 = 0; q2 < Q; ++q2) {
                base[q2] = off[q2];
                cnt[q2] = q2 == q ? 0 : off[q2 + 1] - off[q2];
            }
            for (int it = 0; it < steps; ++it)
#pragma unroll
                for (int q2 = 0; q2 < Q; ++q2)
                    if (cnt[q2] > 0) {
                        const int32_t half = cnt[q2] >> 1;
                        if (si[base[q2] + half] < idx) {
                            base[q2] += half + 1;
                            cnt[q2] -= half + 1;
                        } else {
                            cnt[q2] = half;
                        }
                    }
            int32_t r = e - off[q];
#pragma unroll
            for (int q2 = 0; q2 < Q; ++q2) r += base[q2] - off[q2];
            m_idx[mo + r] = idx;
            m_t[mo + r] = s_t[w][e];
            m_q[mo + r] = (uint8_t)q;
        }
    }
    __syncthreads();
    if (staged)  // decay factors: T is the previous event's time, 0 before the first
        for (int32_t r = lane; r < L; r += kLifThreads) {
            const double ti = (double)m_t[mo + r];
            const double T = r > 0 ? (double)m_t[mo + r - 1] : 0.0;
            m_e[mo + r] = exp(-(ti - T) / A.decay);
        }
    __syncthreads();
    if (w == 0) {
        // the recursions of the block's staged cells, a lane each; a spike
        // marks its merged entry (bit 7 of m_q) and the flags are written
        // after.  Operands come a chunk ahead: m_e and m_q of chunk c+1 are
        // read while chunk c runs, and its 1/n from them one chunk later;
        // reads past a cell's end are clamped into the array and unused.
        const int g = lane;
        const bool mine = g < C && (int64_t)blockIdx.x * C + g < cells && s_moff[g] >= 0;
        const int32_t go = mine ? s_moff[g] : 0, gL = mine ? s_L[g] : 0;
        const int gg = g < C ? g : 0;
        constexpr int kC = 8;
        auto at = [&](int32_t r) { return go + r < MG ? go + r : MG - 1; };
        auto inc_of = [&](int q) { return s_inc[gg][q < Q ? q : 0]; };
        double e_c[kC], i_c[kC], e_n[kC];
        int q_n[kC];
#pragma unroll
        for (int u = 0; u < kC; ++u) {
            e_c[u] = m_e[at(u)];
            i_c[u] = inc_of(m_q[at(u)]);
            q_n[u] = m_q[at(kC + u)];
            e_n[u] = m_e[at(kC + u)];
        }
        double V = 0.0;
        for (int32_t r0 = 0; r0 < gL; r0 += kC) {
            double i_n[kC], e_nn[kC];
            int q_nn[kC];
#pragma unroll
            for (int u = 0; u < kC; ++u) {
                i_n[u] = inc_of(q_n[u]);
                q_nn[u] = m_q[at(r0 + 2 * kC + u)];
                e_nn[u] = m_e[at(r0 + 2 * kC + u)];
            }
#pragma unroll
            for (int u = 0; u < kC; ++u) {
                if (r0 + u < gL) {
                    const double v = V * e_c[u] + i_c[u];
                    const bool fire = v > A.thresh;
                    V = fire ? A.reset : v;
                    if (fire) m_q[go + r0 + u] |= 0x80;
                }
            }
#pragma unroll
            for (int u = 0; u < kC; ++u) {
                e_c[u] = e_n[u];
                i_c[u] = i_n[u];
                e_n[u] = e_nn[u];
                q_n[u] = q_nn[u];
            }
        }
    } else if (lane == 0) {
        // cells beyond the staging run alone, one lane each, on the other waves
        for (int g = w - 1; g < C; g += C - 1) {
            const int64_t c = (int64_t)blockIdx.x * C + g;
            if (c < cells && s_moff[g] < 0)
                cell_sequential<K>(A, (int32_t)(c % A.Wo), (int32_t)(c / A.Wo));
        }
    }
    __syncthreads();
    if (staged)  // the spikes of this wave's cell
        for (int32_t r = lane; r < L; r += kLifThreads) {
            const int q = m_q[mo + r];
            if (q & 0x80)
                mark_spike(A, m_idx[mo + r], s_slot[w][q & 0x7f]);
        }
}

// One thread per (event, slot): the spikes, in scan order.
__global__ void lif_emit_kernel(LifArgs A, const int32_t *__restrict__ flags,
                                const int32_t *__restrict__ place, const int32_t *__restrict__ t,
                                int64_t capacity, int32_t *__restrict__ out_x,
                                int32_t *__restrict__ out_y, int32_t *__restrict__ out_t,
                                int32_t *__restrict__ out_src) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t nslots = (int64_t)A.nsd * A.nsd;
    if (e >= (int64_t)A.n * nslots || !flags[e]) return;
    const int64_t o = place[e];
    if (o >= capacity) return;
    const int32_t i = (int32_t)(e / nslots), s = (int32_t)(e % nslots);
    int32_t lx, hx, ly, hy;
    cell_range(A.px[i], A, A.Wo, lx, hx);
    cell_range(A.py[i], A, A.Ho, ly, hy);
    out_x[o] = lx + s % A.nsd;
    out_y[o] = ly + s / A.nsd;
    out_t[o] = t[i];
    if (out_src) out_src[o] = i;
}

struct LifWs {
    PixelLists pl;
    int32_t *flags, *fpos;
    int64_t *total;
    uint32_t *status;
    void *scan_ws;
};

int32_t lif_slots(int32_t kernel, int32_t stride) {
    const int32_t nsd = (kernel - 1) / stride + 1;
    return nsd * nsd;
}

LifWs carve_lif(void *base, int32_t n, int64_t npix, int64_t nflags, size_t *bytes) {
    Carver cv(base);
    LifWs w;
    w.pl = carve_pixel_lists(cv, n, npix);
    w.flags = cv.take<int32_t>(nflags);
    w.fpos = cv.take<int32_t>(nflags + 1);
    w.total = cv.take<int64_t>(2);
    w.status = cv.take<uint32_t>(4);
    w.scan_ws = cv.take<char>(scan_workspace_bytes(nflags));
    if (bytes) *bytes = cv.used;
    return w;
}

sbc_status check_lif_shape(int32_t n, int32_t width, int32_t height, int32_t kernel,
                           int32_t stride) {
    if (n < 0 || width <= 0 || height <= 0)
        return fail(SBC_ERR_INVALID_ARG, "n must be >= 0, width and height > 0");
    if ((int64_t)width * height >= (int64_t)INT32_MAX)
        return fail(SBC_ERR_INVALID_ARG, "width * height must be < 2^31 - 1");
    if (kernel < 1 || kernel > kLifMaxKernel)
        return fail(SBC_ERR_UNSUPPORTED, "kernel must be 1..5");
    if (stride < 1) return fail(SBC_ERR_INVALID_ARG, "stride must be >= 1");
    if ((int64_t)n * lif_slots(kernel, stride) >= (int64_t)INT32_MAX)
        return fail(SBC_ERR_OVERFLOW, "n * cells reached per event must be < 2^31 - 1");
    return SBC_OK;
}

}  // namespace
}  // namespace sbc

using namespace sbc;

extern "C" size_t sbc_lif_workspace_size(int32_t n, int32_t width, int32_t height,
                                         int32_t kernel, int32_t stride) {
    if (check_lif_shape(n, width, height, kernel, stride) != SBC_OK) {
        clear_error();
        return 0;
    }
    size_t bytes = 0;
    carve_lif(nullptr, n, (int64_t)width * height, (int64_t)n * lif_slots(kernel, stride),
              &bytes);
    return bytes;
}

extern "C" sbc_status sbc_lif_sample_events(const int32_t *px, const int32_t *py,
                                            const int32_t *t, int32_t n, int32_t width,
                                            int32_t height, int32_t kernel, int32_t stride,
                                            double decay, double v_thresh, double v_reset,
                                            int32_t *out_x, int32_t *out_y, int32_t *out_t,
                                            int32_t *out_src, int64_t capacity,
                                            int64_t *n_out_dev, int64_t *n_out_host,
                                            void *workspace, size_t workspace_bytes,
                                            hipStream_t stream) {
    clear_error();
    SBC_TRY(check_lif_shape(n, width, height, kernel, stride));
    if (!(decay > 0.0)) return fail(SBC_ERR_INVALID_ARG, "decay must be > 0 (inf: no decay)");
    if (n > 0 && (!px || !py || !t)) return fail(SBC_ERR_INVALID_ARG, "null event arrays");
    if (capacity < 0 || (capacity > 0 && (!out_x || !out_y || !out_t)))
        return fail(SBC_ERR_INVALID_ARG, "output arrays are null, or capacity < 0");
    const int64_t npix = (int64_t)width * height;
    const int32_t slots = lif_slots(kernel, stride);
    const int64_t nflags = (int64_t)n * slots;
    size_t need = 0;
    LifWs ws = carve_lif(workspace, n, npix, nflags, &need);
    if (!workspace || workspace_bytes < need)
        return fail(SBC_ERR_WORKSPACE, "workspace smaller than sbc_lif_workspace_size()");
    LifArgs A{};
    A.px = px;
    A.py = py;
    A.n = n;
    A.W = width;
    A.H = height;
    A.S = stride;
    A.k = kernel;
    A.pad = (kernel - 1) / 2;
    A.Wo = (width + stride - 1) / stride;
    A.Ho = (height + stride - 1) / stride;
    A.nsd = (kernel - 1) / stride + 1;
    A.decay = decay;
    A.thresh = v_thresh;
    A.reset = v_reset;
    A.pix_start = ws.pl.pix_start;
    A.list = ws.pl.list;
    A.list_t = ws.pl.list_t;
    A.flags = ws.flags;
    A.status = ws.status;
    int64_t *total = n_out_dev ? n_out_dev : ws.total;

    SBC_TRY(fill_i32(reinterpret_cast<int32_t *>(ws.status), 0, 1, stream));
    if (n > 0) {
        trace_before("lif_sort", stream);
        SBC_TRY(build_pixel_lists(px, py, t, n, width, height, ws.pl, ws.status, ws.flags, slots,
                                  stream));
        trace_after("lif_sort", stream);
        const int64_t cells = (int64_t)A.Wo * A.Ho;
        trace_before("lif_cells", stream);
#define SBC_LIF_CELLS(KK)                                                                      \
    hipLaunchKernelGGL(lif_cell_kernel<KK>, dim3(grid_for(cells, LifTile<KK>::kCells)),      \
                       dim3(LifTile<KK>::kCells * kLifThreads), 0, stream, A)
        switch (kernel) {
            case 1: SBC_LIF_CELLS(1); break;
            case 2: SBC_LIF_CELLS(2); break;
            case 3: SBC_LIF_CELLS(3); break;
            case 4: SBC_LIF_CELLS(4); break;
            default: SBC_LIF_CELLS(5); break;
        }
#undef SBC_LIF_CELLS
        SBC_LAUNCH_CHECK();
        trace_after("lif_cells", stream);
    }
    SBC_TRY(exclusive_scan_i32(ws.flags, ws.fpos, nflags, total, ws.scan_ws, stream));
    if (nflags > 0 && capacity > 0) {
        trace_before("lif_emit", stream);
        hipLaunchKernelGGL(lif_emit_kernel, dim3(grid_for(nflags, 256)), dim3(256), 0, stream, A,
                           ws.flags, ws.fpos, t, capacity, out_x, out_y, out_t, out_src);
        SBC_LAUNCH_CHECK();
        trace_after("lif_emit", stream);
    }
    if (n_out_host) {
        int64_t count = 0;
        uint32_t st = 0;
        SBC_HIP_TRY(hipMemcpyAsync(&count, total, sizeof(count), hipMemcpyDeviceToHost, stream));
        SBC_HIP_TRY(hipMemcpyAsync(&st, ws.status, sizeof(st), hipMemcpyDeviceToHost, stream));
        SBC_HIP_TRY(hipStreamSynchronize(stream));
        *n_out_host = count;
        if (st & kFlagInternal)
            return fail(SBC_ERR_INTERNAL, "a spike flag index fell outside the flags");
        if (st & kFlagOutOfRange) return fail(SBC_ERR_OUT_OF_RANGE, "pixel outside the sensor");
        if (st & kFlagUnsorted) return fail(SBC_ERR_UNSORTED, "timestamps must be non-decreasing");
        if (count > capacity)
            return fail(SBC_ERR_CAPACITY, "capacity " + std::to_string(capacity) +
                                              " < output events " + std::to_string(count));
    }
    return SBC_OK;
}
