// Internal helpers shared by the sbconv HIP sources: error state, workspace
// carving, launch checks, small device utilities.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <string>

#include "../../include/sbconv.h"

namespace sbc {

// ---------------------------------------------------------------- errors
void set_error(const std::string &msg);
void clear_error();
sbc_status fail(sbc_status st, const std::string &msg);

#define SBC_HIP_TRY(expr)                                                              \
    do {                                                                               \
        hipError_t _e = (expr);                                                        \
        if (_e != hipSuccess)                                                          \
            return ::sbc::fail(SBC_ERR_HIP, std::string(#expr) + ": " +                \
                                                hipGetErrorString(_e));                \
    } while (0)

#define SBC_LAUNCH_CHECK()                                                             \
    do {                                                                               \
        hipError_t _e = hipGetLastError();                                             \
        if (_e != hipSuccess)                                                          \
            return ::sbc::fail(SBC_ERR_HIP, std::string("kernel launch: ") +           \
                                                hipGetErrorString(_e));                \
    } while (0)

#define SBC_TRY(expr)                                                                  \
    do {                                                                               \
        sbc_status _s = (expr);                                                        \
        if (_s != SBC_OK) return _s;                                                   \
    } while (0)

// ---------------------------------------------------------------- tracing
// Record the caller's events around launches of the kernel `name` (no-op
// unless sbc_trace_kernel registered that name on this thread).
void trace_before(const char *name, hipStream_t stream);
void trace_after(const char *name, hipStream_t stream);

// ---------------------------------------------------------------- workspace
constexpr size_t kAlign = 256;

inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Hands out 256-byte aligned slices of one caller-provided buffer.  With a
// null base it only measures.
struct Carver {
    char *base;
    size_t used = 0;
    explicit Carver(void *b) : base(static_cast<char *>(b)) {}
    template <typename T> T *take(size_t count) {
        size_t off = used;
        used += align_up(count * sizeof(T) + 1);
        return base ? reinterpret_cast<T *>(base + off) : nullptr;
    }
};

// ---------------------------------------------------------------- device status word
// Bits a kernel may raise in a device-side status word (the host reads the
// word back only where an entry point synchronises anyway).
enum : uint32_t {
    kFlagOutOfRange = 1u,
    kFlagUnsorted = 2u,
    kFlagCapacity = 4u,
    kFlagBadSplits = 8u,
    kFlagInternal = 16u,  // a kernel's own index check failed (its store was skipped)
};

// ---------------------------------------------------------------- primitives (scan.hip)
// Exclusive prefix sum of `n` int32 counts into out[0..n]; out[n] is the total.
// The total is also stored, as int64, to *total64 (device, may be null).  Sums
// of 2^31 or more are saturated in `out` and still exact in *total64.  out2
// (may be null) receives a second copy of out.  Short arrays take one kernel.
size_t scan_workspace_bytes(int64_t n);
sbc_status exclusive_scan_i32(const int32_t *counts, int32_t *out, int64_t n, int64_t *total64,
                              void *ws, hipStream_t stream, int32_t *out2 = nullptr);
// Exclusive scans of two arrays of n items (a into a_out, b into b_out, each
// with its total at [n]) in one pair of launches; workspace
// scan2_workspace_bytes(n).
size_t scan2_workspace_bytes(int64_t n);
sbc_status exclusive_scan2_i32(const int32_t *a, int32_t *a_out, const int32_t *b,
                               int32_t *b_out, int64_t n, int64_t *a_total64,
                               int64_t *b_total64, void *ws, hipStream_t stream);

// Fill n int32 words with a value (a kernel, not a memset node).
sbc_status fill_i32(int32_t *p, int32_t value, int64_t n, hipStream_t stream);

// Sort the entries of each segment [ptr[s], ptr[s+1]) of (key, payload) pairs by
// key ascending (keys distinct within a segment), writing to the *_out arrays.
// seg_of[p] is the segment of entry p; only entries p < min(ptr[n_segments],
// n_bound) are sorted.  val_in / val_out may be null (keys only).
sbc_status segmented_sort_pairs(const int32_t *ptr, int32_t n_segments, const int32_t *seg_of,
                                int64_t n_bound, const int32_t *key_in, const int32_t *val_in,
                                int32_t *key_out, int32_t *val_out, hipStream_t stream);

// Stable radix sort (sort.hip) of n (key, value) pairs, keys in [0, key_bound);
// n = *n_dev clamped to [0, n_bound] (n_dev may be null: n = n_bound).
// vals == nullptr: the values are the item indices.  No global atomics.
size_t radix_sort_workspace_bytes(int64_t n_bound);
sbc_status radix_sort_pairs(const int32_t *keys, const int32_t *vals, const int64_t *n_dev,
                            int64_t n_bound, int32_t key_bound, int32_t *keys_out,
                            int32_t *vals_out, void *ws, hipStream_t stream);
// ptr[k] = first position of the sorted keys with key >= k, for k in
// [0, key_bound]; keys must lie in [0, key_bound].
sbc_status segment_bounds(const int32_t *sorted, const int64_t *n_dev, int64_t n_bound,
                          int32_t key_bound, int32_t *ptr, hipStream_t stream);

// Compute units of the current device (256 if the query fails); sizes
// persistent grids.
int device_cus();

inline int grid_for(int64_t n, int block) {
    int64_t g = (n + block - 1) / block;
    return static_cast<int>(g < 1 ? 1 : g);
}

}  // namespace sbc
