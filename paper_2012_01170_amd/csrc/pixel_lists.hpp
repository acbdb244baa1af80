// Per-pixel lists of an event stream, each in stream order with the events'
// times alongside (pixel_lists.hip): shared by the stream samplers.
#pragma once

#include "common.hpp"

namespace sbc {

struct PixelLists {
    int32_t *pix_start;  // [npix + 1]: pixel p's events are list[pix_start[p] ..)
    int32_t *list;       // [n] event indices (the first pix_start[npix] are listed)
    int32_t *list_t;     // [n] their times
    int32_t *counts, *keys, *place, *unsorted, *unsorted_t, *seg_of;
    int64_t *total;
    void *scan_ws;
};

PixelLists carve_pixel_lists(Carver &cv, int32_t n, int64_t npix);

// Builds the lists: a count with integer atomics (raising kFlagOutOfRange for
// an event off the sensor, which is not listed, and kFlagUnsorted for
// decreasing times in *status), a scan, a placement, and a rank sort inside
// each pixel's segment.  The count kernel also zeroes clear[0 .. n * per_event)
// (clear may be null).  n >= 1.
sbc_status build_pixel_lists(const int32_t *px, const int32_t *py, const int32_t *t, int32_t n,
                             int32_t W, int32_t H, const PixelLists &pl, uint32_t *status,
                             int32_t *clear, int32_t per_event, hipStream_t stream);

}  // namespace sbc
