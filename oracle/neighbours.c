/*
 * CPU ORACLE -- test infrastructure only.  Nothing in the product library
 * links, includes or calls this file; only the tests, the smoke check and the
 * benchmark's CPU-baseline leg load it.
 *
 * Neighbour sets of the sparse basis convolution, enumerated exhaustively.
 *
 * Points (Section 3.1, "Neighborhoods"; the ball of radius r, optionally
 * truncated to the k nearest members): output point i of cloud b has as
 * neighbours the inputs j of the same cloud with d2(x'_i, x_j) < r*r, where d2
 * is evaluated in float32, round to nearest, no fused multiply-add, as
 *     dx = x'.x - x.x  (same for y, z);  d2 = ((dx*dx) + (dy*dy)) + (dz*dz).
 * With k_cap > 0 and more than k_cap members, the k_cap smallest by (d2, j)
 * are kept.  Each row is emitted in ascending j.  Ragged batches are the
 * block-diagonal concatenation of clouds (Section 3.1, "Ragged Batching").
 *
 * Events (Section 3.2, the event kernel and its backwards-in-time domain):
 * event i has as neighbours the earlier events j < i whose pixel lies within
 * the (2h+1)x(2h+1) block around its own, |px_i - px_j| <= h and
 * |py_i - py_j| <= h, and with t_i - t_j <= window.  Timestamps are integer
 * and non-decreasing in stream order.
 *
 * Build: gcc -O2 -std=c99 -ffp-contract=off -fopenmp -shared -fPIC.
 * The OpenMP loops run independent rows in parallel; each row is computed
 * exactly as the serial definition would.
 */
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Number of threads the parallel loops below use. */
int orc_max_threads(void) { return omp_get_max_threads(); }

typedef struct {
    float d2;
    int32_t j;
} cand_t;

static int cmp_d2_j(const void *a, const void *b) {
    const cand_t *x = (const cand_t *)a, *y = (const cand_t *)b;
    if (x->d2 < y->d2) return -1;
    if (x->d2 > y->d2) return 1;
    return (x->j > y->j) - (x->j < y->j);
}

static int cmp_j(const void *a, const void *b) {
    const cand_t *x = (const cand_t *)a, *y = (const cand_t *)b;
    return (x->j > y->j) - (x->j < y->j);
}

static float sq_dist_f32(const float *p, const float *q) {
    volatile float dx = p[0] - q[0];
    volatile float dy = p[1] - q[1];
    volatile float dz = p[2] - q[2];
    volatile float xx = dx * dx;
    volatile float yy = dy * dy;
    volatile float zz = dz * dz;
    volatile float s = xx + yy;
    return s + zz;
}

/* Cloud index of output row i (out_splits is non-decreasing, n_batch + 1 long). */
static int cloud_of(const int32_t *splits, int n_batch, int32_t i) {
    int b = 0;
    while (b + 1 < n_batch && splits[b + 1] <= i) ++b;
    return b;
}

/*
 * Row i of the point CSR.  Writes its column indices to `out` (may be NULL)
 * and returns the row length.
 */
static int32_t point_row(const float *x_in, const int32_t *in_splits, const float *x_out,
                         const int32_t *out_splits, int n_batch, float radius, int32_t k_cap,
                         int32_t i, int32_t *out) {
    int b = cloud_of(out_splits, n_batch, i);
    int32_t j0 = in_splits[b], j1 = in_splits[b + 1];
    volatile float r2 = radius * radius;
    cand_t *c = (cand_t *)malloc(sizeof(cand_t) * (size_t)(j1 - j0 + 1));
    int32_t n = 0;
    for (int32_t j = j0; j < j1; ++j) {
        float d2 = sq_dist_f32(x_out + 3 * (size_t)i, x_in + 3 * (size_t)j);
        if (d2 < r2) {
            c[n].d2 = d2;
            c[n].j = j;
            ++n;
        }
    }
    if (k_cap > 0 && n > k_cap) {
        qsort(c, (size_t)n, sizeof(cand_t), cmp_d2_j);
        n = k_cap;
    }
    qsort(c, (size_t)n, sizeof(cand_t), cmp_j);
    if (out)
        for (int32_t q = 0; q < n; ++q) out[q] = c[q].j;
    free(c);
    return n;
}

static int64_t finish_row_ptr(int32_t *row_ptr, int32_t n_rows) {
    int64_t acc = 0;
    for (int32_t i = 0; i < n_rows; ++i) {
        int64_t len = row_ptr[i + 1];
        row_ptr[i] = (int32_t)acc;
        acc += len;
    }
    row_ptr[n_rows] = (int32_t)acc;
    return acc;
}

/*
 * Pass 1 (col_idx == NULL): fills row_ptr[0..n_out] and returns E.
 * Pass 2 (col_idx != NULL, row_ptr from pass 1): fills col_idx, returns E.
 */
int64_t orc_points_brute(const float *x_in, const int32_t *in_splits, const float *x_out,
                         const int32_t *out_splits, int32_t n_batch, int32_t n_out,
                         float radius, int32_t k_cap, int32_t *row_ptr, int32_t *col_idx) {
    if (!col_idx) {
#pragma omp parallel for schedule(dynamic, 16)
        for (int32_t i = 0; i < n_out; ++i)
            row_ptr[i + 1] = point_row(x_in, in_splits, x_out, out_splits, n_batch, radius,
                                       k_cap, i, NULL);
        return finish_row_ptr(row_ptr, n_out);
    }
#pragma omp parallel for schedule(dynamic, 16)
    for (int32_t i = 0; i < n_out; ++i)
        point_row(x_in, in_splits, x_out, out_splits, n_batch, radius, k_cap, i,
                  col_idx + row_ptr[i]);
    return row_ptr[n_out];
}

/* Same, also returning the fp32 d2 of each kept edge (used by tests of the cap). */
int64_t orc_points_d2(const float *x_in, const float *x_out, const int32_t *row_ptr,
                      const int32_t *col_idx, int32_t n_out, float *d2_out) {
    for (int32_t i = 0; i < n_out; ++i)
        for (int32_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e)
            d2_out[e] = sq_dist_f32(x_out + 3 * (size_t)i, x_in + 3 * (size_t)col_idx[e]);
    return row_ptr[n_out];
}

static int event_pair(const int32_t *px, const int32_t *py, const int32_t *t, int32_t i,
                      int32_t j, int32_t h, int32_t window) {
    int32_t ax = px[i] - px[j], ay = py[i] - py[j];
    if (ax < 0) ax = -ax;
    if (ay < 0) ay = -ay;
    return ax <= h && ay <= h && (int64_t)t[i] - (int64_t)t[j] <= (int64_t)window;
}

/*
 * Every earlier event j < i is tested (quadratic; for small streams).
 * Two passes as for points.
 */
int64_t orc_events_quadratic(const int32_t *px, const int32_t *py, const int32_t *t, int32_t n,
                             int32_t h, int32_t window, int32_t *row_ptr, int32_t *col_idx) {
#pragma omp parallel for schedule(dynamic, 64)
    for (int32_t i = 0; i < n; ++i) {
        int32_t cnt = 0;
        int32_t base = col_idx ? row_ptr[i] : 0;
        for (int32_t j = 0; j < i; ++j)
            if (event_pair(px, py, t, i, j, h, window)) {
                if (col_idx) col_idx[base + cnt] = j;
                ++cnt;
            }
        if (!col_idx) row_ptr[i + 1] = cnt;
    }
    return col_idx ? row_ptr[n] : finish_row_ptr(row_ptr, n);
}

/*
 * Windowed scan: because t is non-decreasing, the earlier events with
 * t_i - t_j <= window are exactly a contiguous run j = lo(i) .. i-1; each of
 * them is tested.
 */
int64_t orc_events_scan(const int32_t *px, const int32_t *py, const int32_t *t, int32_t n,
                        int32_t h, int32_t window, int32_t *row_ptr, int32_t *col_idx) {
#pragma omp parallel for schedule(dynamic, 64)
    for (int32_t i = 0; i < n; ++i) {
        int32_t lo = i;
        while (lo > 0 && (int64_t)t[i] - (int64_t)t[lo - 1] <= (int64_t)window) --lo;
        int32_t cnt = 0;
        int32_t base = col_idx ? row_ptr[i] : 0;
        for (int32_t j = lo; j < i; ++j)
            if (event_pair(px, py, t, i, j, h, window)) {
                if (col_idx) col_idx[base + cnt] = j;
                ++cnt;
            }
        if (!col_idx) row_ptr[i + 1] = cnt;
    }
    return col_idx ? row_ptr[n] : finish_row_ptr(row_ptr, n);
}

/*
 * Per-pixel lists: every pixel keeps the indices of its events in stream
 * order; event i visits the (2h+1)^2 pixels around it and walks each list back
 * from the last event before i while the time gap stays within the window.
 * The visited indices are gathered and sorted ascending.
 */
int64_t orc_events_pixels(const int32_t *px, const int32_t *py, const int32_t *t, int32_t n,
                          int32_t width, int32_t height, int32_t h, int32_t window,
                          int32_t *row_ptr, int32_t *col_idx) {
    int64_t npix = (int64_t)width * height;
    int32_t *start = (int32_t *)calloc((size_t)npix + 1, sizeof(int32_t));
    int32_t *list = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
    for (int32_t i = 0; i < n; ++i) start[(int64_t)py[i] * width + px[i] + 1]++;
    for (int64_t p = 0; p < npix; ++p) start[p + 1] += start[p];
    {
        int32_t *fill = (int32_t *)malloc(sizeof(int32_t) * (size_t)(npix > 0 ? npix : 1));
        memcpy(fill, start, sizeof(int32_t) * (size_t)npix);
        for (int32_t i = 0; i < n; ++i) {
            int64_t p = (int64_t)py[i] * width + px[i];
            list[fill[p]++] = i;
        }
        free(fill);
    }
#pragma omp parallel for schedule(dynamic, 256)
    for (int32_t i = 0; i < n; ++i) {
        int32_t buf_cap = 64, cnt = 0;
        int32_t *buf = (int32_t *)malloc(sizeof(int32_t) * (size_t)buf_cap);
        for (int32_t qy = py[i] - h; qy <= py[i] + h; ++qy) {
            if (qy < 0 || qy >= height) continue;
            for (int32_t qx = px[i] - h; qx <= px[i] + h; ++qx) {
                if (qx < 0 || qx >= width) continue;
                int64_t p = (int64_t)qy * width + qx;
                /* position in list p of the last event with index < i */
                int32_t a = start[p], b = start[p + 1];
                int32_t lo = a, hi = b; /* first position with list[pos] >= i */
                while (lo < hi) {
                    int32_t mid = lo + (hi - lo) / 2;
                    if (list[mid] < i) lo = mid + 1; else hi = mid;
                }
                for (int32_t pos = lo - 1; pos >= a; --pos) {
                    int32_t j = list[pos];
                    if ((int64_t)t[i] - (int64_t)t[j] > (int64_t)window) break;
                    if (cnt == buf_cap) {
                        buf_cap *= 2;
                        buf = (int32_t *)realloc(buf, sizeof(int32_t) * (size_t)buf_cap);
                    }
                    buf[cnt++] = j;
                }
            }
        }
        if (col_idx) {
            /* insertion sort ascending */
            for (int32_t a2 = 1; a2 < cnt; ++a2) {
                int32_t v = buf[a2], b2 = a2 - 1;
                while (b2 >= 0 && buf[b2] > v) { buf[b2 + 1] = buf[b2]; --b2; }
                buf[b2 + 1] = v;
            }
            memcpy(col_idx + row_ptr[i], buf, sizeof(int32_t) * (size_t)cnt);
        } else {
            row_ptr[i + 1] = cnt;
        }
        free(buf);
    }
    free(list);
    free(start);
    return col_idx ? row_ptr[n] : finish_row_ptr(row_ptr, n);
}

/* Stable transpose by counting sort on the column (rows stay ascending). */
void orc_csr_transpose(const int32_t *row_ptr, const int32_t *col_idx, int32_t n_rows,
                       int32_t n_cols, int32_t *col_ptr, int32_t *row_idx, int32_t *edge_perm) {
    memset(col_ptr, 0, sizeof(int32_t) * ((size_t)n_cols + 1));
    int64_t E = row_ptr[n_rows];
    for (int64_t e = 0; e < E; ++e) col_ptr[col_idx[e] + 1]++;
    for (int32_t c = 0; c < n_cols; ++c) col_ptr[c + 1] += col_ptr[c];
    int32_t *fill = (int32_t *)malloc(sizeof(int32_t) * ((size_t)n_cols + 1));
    memcpy(fill, col_ptr, sizeof(int32_t) * ((size_t)n_cols + 1));
    for (int32_t i = 0; i < n_rows; ++i)
        for (int32_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
            int32_t pos = fill[col_idx[e]]++;
            row_idx[pos] = i;
            edge_perm[pos] = e;
        }
    free(fill);
}
