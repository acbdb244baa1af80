// Per-pixel event lists in stream order (see pixel_lists.hpp).
#include "pixel_lists.hpp"

namespace sbc {
namespace {

// Each event's pixel, counted; the atomic's value is the event's provisional
// place in its pixel's list (sorted by index afterwards).
__global__ void pixel_count_kernel(const int32_t *__restrict__ px, const int32_t *__restrict__ py,
                                   const int32_t *__restrict__ t, int32_t n, int32_t W, int32_t H,
                                   int32_t per_event, int32_t *__restrict__ clear,
                                   int32_t *__restrict__ counts, int32_t *__restrict__ keys,
                                   int32_t *__restrict__ place, uint32_t *status) {
    const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    if (clear)
        for (int32_t s = 0; s < per_event; ++s) clear[(int64_t)i * per_event + s] = 0;
    const int32_t x = px[i], y = py[i];
    if (i > 0 && t[i] < t[i - 1]) atomicOr(status, (uint32_t)kFlagUnsorted);
    if (x < 0 || x >= W || y < 0 || y >= H) {
        atomicOr(status, (uint32_t)kFlagOutOfRange);
        keys[i] = -1;  // not listed
        return;
    }
    const int32_t p = y * W + x;
    keys[i] = p;
    place[i] = atomicAdd(&counts[p], 1);
}

// Each listed event to a place of its pixel's list, with its time.
__global__ void pixel_place_kernel(const int32_t *__restrict__ keys,
                                   const int32_t *__restrict__ place,
                                   const int32_t *__restrict__ pix_start,
                                   const int32_t *__restrict__ t, int32_t n,
                                   int32_t *__restrict__ unsorted,
                                   int32_t *__restrict__ unsorted_t,
                                   int32_t *__restrict__ seg_of) {
    const int32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n || keys[i] < 0) return;
    const int32_t p = keys[i];
    const int32_t pos = pix_start[p] + place[i];
    unsorted[pos] = i;
    unsorted_t[pos] = t[i];
    seg_of[pos] = p;
}

}  // namespace

PixelLists carve_pixel_lists(Carver &cv, int32_t n, int64_t npix) {
    PixelLists pl;
    pl.counts = cv.take<int32_t>(npix);
    pl.keys = cv.take<int32_t>(n);
    pl.place = cv.take<int32_t>(n);
    pl.unsorted = cv.take<int32_t>(n);
    pl.unsorted_t = cv.take<int32_t>(n);
    pl.seg_of = cv.take<int32_t>(n);
    pl.list = cv.take<int32_t>(n);
    pl.list_t = cv.take<int32_t>(n);
    pl.pix_start = cv.take<int32_t>(npix + 1);
    pl.total = cv.take<int64_t>(2);
    pl.scan_ws = cv.take<char>(scan_workspace_bytes(npix));
    return pl;
}

sbc_status build_pixel_lists(const int32_t *px, const int32_t *py, const int32_t *t, int32_t n,
                             int32_t W, int32_t H, const PixelLists &pl, uint32_t *status,
                             int32_t *clear, int32_t per_event, hipStream_t stream) {
    const int64_t npix = (int64_t)W * H;
    const dim3 eg(grid_for(n, 256)), eb(256);
    SBC_TRY(fill_i32(pl.counts, 0, npix, stream));
    hipLaunchKernelGGL(pixel_count_kernel, eg, eb, 0, stream, px, py, t, n, W, H, per_event,
                       clear, pl.counts, pl.keys, pl.place, status);
    SBC_LAUNCH_CHECK();
    SBC_TRY(exclusive_scan_i32(pl.counts, pl.pix_start, npix, pl.total, pl.scan_ws, stream));
    hipLaunchKernelGGL(pixel_place_kernel, eg, eb, 0, stream, pl.keys, pl.place, pl.pix_start, t,
                       n, pl.unsorted, pl.unsorted_t, pl.seg_of);
    SBC_LAUNCH_CHECK();
    // each pixel's list in stream order (indices are distinct), times alongside
    return segmented_sort_pairs(pl.pix_start, (int32_t)npix, pl.seg_of, n, pl.unsorted,
                                pl.unsorted_t, pl.list, pl.list_t, stream);
}

}  // namespace sbc
