/*
 * sbconv -- sparse basis convolution on continuous domains (point clouds and
 * event streams), after "Sparse Convolutions on Continuous Domains for Point
 * Cloud and Event Stream Networks" (Jack, Maire, Denman, Eriksson, ACCV 2020).
 *
 * The operator (Section 3.1, the matrix-product form of the convolution):
 *
 *     Y = sum_m  N^(m) F W^(m)
 *
 *   F    [n_in,  C_in ]  features of the input points / events
 *   W    [M, C_in, C_out] learned weights, one C_in x C_out matrix per basis fn
 *   N^(m)[n_out, n_in]   sparse neighbourhood matrices sharing one pattern:
 *                        entry (i, j) = p_m(x'_i - x_j) for j in the
 *                        neighbourhood of output i, zero otherwise
 *   Y    [n_out, C_out]
 *
 * Conventions of every entry point
 *   - Array arguments are DEVICE pointers unless their name ends in _host.
 *   - Every array is row-major and densely packed.  Buffers are owned by the
 *     caller; the library keeps no pointer after a call returns and allocates
 *     no device memory: temporary space comes from the `workspace` argument,
 *     whose required size a *_workspace_size query gives.  workspace must be
 *     256-byte aligned; the feature, weight, output and gradient arrays of the
 *     convolution calls 16-byte aligned (rows move 16 bytes at a time).
 *   - Work is enqueued on `stream` and runs asynchronously; only a neighbour
 *     search given a non-NULL nnz_host synchronises the stream (once).
 *   - Outputs are overwritten, never accumulated into.
 *   - Indices are int32; an edge count of 2^31 or more is an error.
 *   - On an argument error nothing is enqueued and a status other than
 *     SBC_OK is returned; sbc_last_error() then describes it (thread-local).
 *   - Results are deterministic: no floating-point atomics are used, so the
 *     same inputs give bitwise-identical outputs on every run.
 *
 * CSR layout of the neighbourhoods: rows are outputs i, row_ptr [n_out + 1],
 * col_idx [E] holds input indices j: ascending within a row for point
 * patterns, in block order for event patterns (section 1b).  The matrix is
 * defined entry by entry, so the order within a row only fixes the order in
 * which the kernels add up a row's terms.  A ragged batch
 * of clouds is the block-diagonal matrix of the per-cloud matrices with
 * global column indices (Section 3.1, "Ragged Batching").
 */
#ifndef SBCONV_H
#define SBCONV_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    SBC_OK = 0,
    SBC_ERR_INVALID_ARG = 1,  /* null pointer, bad size, unknown enum, ...        */
    SBC_ERR_CAPACITY = 2,     /* col_idx too small for the edges found            */
    SBC_ERR_OVERFLOW = 3,     /* 2^31 or more edges                               */
    SBC_ERR_UNSORTED = 4,     /* event timestamps decrease somewhere              */
    SBC_ERR_OUT_OF_RANGE = 5, /* pixel outside the sensor, split outside [0, n]   */
    SBC_ERR_WORKSPACE = 6,    /* workspace smaller than the size query's answer   */
    SBC_ERR_HIP = 7,          /* a HIP runtime call failed                        */
    SBC_ERR_UNSUPPORTED = 8,  /* shape or basis with no kernel in the library    */
    SBC_ERR_INTERNAL = 9      /* a kernel's own consistency check failed; its    */
                              /* stores were skipped (a library defect)           */
} sbc_status;

typedef enum {
    SBC_F32 = 0,  /* float32 features, weights and gradients                    */
    SBC_BF16 = 1  /* bfloat16 features, weights and upstream gradient; float32  */
                  /* basis values, accumulation and outputs                      */
} sbc_dtype;

/*
 * Basis functions p_m.  Point bases (Section 3.1: geometric monomials of the
 * edge vector) use u = (x'_i - x_j) / r and the window w = (1 - |u|^2)^2:
 *   SBC_BASIS_MONO4   M = 4: [1, ux, uy, uz] * w
 *   SBC_BASIS_MONO8   M = 8: [1, ux, uy, uz, ux^2, uy^2, uz^2, ux*uy] * w
 * Event basis (Section 3.2, the event kernel with one decay per pixel offset,
 * lambda = 1/tau): u = (px_i - px_j, py_i - py_j) in the 3x3 block,
 * dt = t_i - t_j >= 0;
 *   SBC_BASIS_EVENT8  M = 8: p_m = [m == idx(u)] * exp(-dt / tau), with idx
 *                     row-major over (uy, ux) and the centre offset removed
 *                     (same-pixel edges have an all-zero basis row).
 * Weighted convolution (Section 3.1, "Weighted Convolutions", Eq. 11) with the
 * full second-order monomial set of the paper's networks, u = (x'_i - x_j) / r:
 *   SBC_BASIS_WMONO10 M = 10: [1, ux, uy, uz, ux^2, uy^2, uz^2, ux*uy, ux*uz,
 *                     uy*uz] * w_ij / W_i, with w_ij = 1 - |x'_i - x_j| / r and
 *                     W_i the sum of w_ij over row i (values 0 if W_i = 0).
 *                     Its values depend on the whole row, so the unfused
 *                     routes evaluate them in CSR order and a transpose given
 *                     to sbc_conv_backward needs its edge_perm.
 * Event kernel with learned decays (Section 3.2, Eq. 12: g(u, dt) =
 * sum_v exp(-lambda_uv dt) theta_uv, M_v decays per offset):
 *   SBC_BASIS_EVENT_DECAYS  M = 8 * n_decays (2 <= n_decays <= 4):
 *                     p_m = [u == idx(offset)] * exp(-lambda_uv * dt) with
 *                     m = u * n_decays + v, u the SBC_BASIS_EVENT8 offset index
 *                     and lambda = geometry.decays[u * n_decays + v] (> 0).
 */
typedef enum {
    SBC_BASIS_MONO4 = 0,
    SBC_BASIS_MONO8 = 1,
    SBC_BASIS_EVENT8 = 2,
    SBC_BASIS_WMONO10 = 3,
    SBC_BASIS_EVENT_DECAYS = 4
} sbc_basis;

/*
 * Evaluation order of the matrix products (Section 3.1, down- vs up-sampling
 * convolutions and their cost table):
 *   SPMM_FIRST  (N^(m) F) W^(m): gather-accumulate G = [N^(0)F ... N^(M-1)F]
 *               [n_out, M*C_in], then one dense contraction with W.
 *   GEMM_FIRST  N^(m) (F W^(m)): one dense contraction H = F [W^(0)..W^(M-1)]
 *               [n_in, M*C_out], then gather-accumulate over H.
 *   AUTO        the library picks by the multiply-add counts of both orders.
 * The backward pass uses the transposed counterpart of the chosen order.
 */
typedef enum {
    SBC_ORDER_AUTO = 0,
    SBC_ORDER_SPMM_FIRST = 1,
    SBC_ORDER_GEMM_FIRST = 2
} sbc_order;

/*
 * The shared sparsity pattern of the N^(m) (rows = outputs).  Kernels read
 * row extents from row_ptr on the device; nnz_bound only sizes per-edge
 * temporaries and must be >= row_ptr[n_rows] (the exact E is best).
 */
typedef struct {
    int32_t n_rows;           /* n_out                                          */
    int32_t n_cols;           /* n_in                                           */
    int64_t nnz_bound;        /* >= E = row_ptr[n_rows]                         */
    const int32_t *row_ptr;   /* [n_rows + 1], row_ptr[0] = 0                   */
    const int32_t *col_idx;   /* [E]                                            */
} sbc_csr;

/* Its transpose (rows = inputs), as produced by sbc_csr_transpose.  edge_perm
 * may be NULL when the basis values are evaluated inside the kernels (v NULL
 * in sbc_conv_backward): they are then evaluated for the transposed entries
 * directly and no entry needs its CSR position. */
typedef struct {
    int32_t n_cols;           /* n_in                                           */
    const int32_t *col_ptr;   /* [n_cols + 1]                                   */
    const int32_t *row_idx;   /* [E] output index of each entry: ascending from
                                 sbc_csr_transpose, in block order from the
                                 event search                                   */
    const int32_t *edge_perm; /* [E] CSR position of each entry, or NULL        */
} sbc_csc;

/*
 * Coordinates the basis values are evaluated from (the paper evaluates the
 * basis on the accelerator from the neighbour indices; Section 3.1, "Data
 * Pipeline").  Point bases read x_in/x_out and radius; the event basis reads
 * px/py/t and tau, for an in-place stream (outputs = inputs).
 */
typedef struct {
    sbc_basis basis;
    float radius;             /* points: r, > 0                                 */
    float tau;                /* events: decay time, > 0, unit of t             */
    const float *x_in;        /* points: [n_in, 3]                              */
    const float *x_out;       /* points: [n_out, 3]                             */
    const int32_t *px;        /* events: [n] pixel column                       */
    const int32_t *py;        /* events: [n] pixel row                          */
    const int32_t *t;         /* events: [n] timestamps, non-decreasing         */
    const float *decays;      /* SBC_BASIS_EVENT_DECAYS: [8, n_decays] rates    */
    int32_t n_decays;         /* SBC_BASIS_EVENT_DECAYS: decays per offset      */
} sbc_geometry;

/* Thread-local description of the last error of this thread ("" if none). */
const char *sbc_last_error(void);
const char *sbc_status_string(sbc_status status);
/* Number of basis functions of a basis (0 for an unknown one). */
int32_t sbc_basis_size(sbc_basis basis);

/* ------------------------------------------------------------------------
 * 1a. Point neighbourhoods (Section 3.1, "Neighborhoods"): for output i of
 * cloud b, the inputs j of cloud b with d2 < r*r, where d2 is evaluated in
 * float32 with round-to-nearest and no fused multiply-add as
 *     dx = x'_i.x - x_j.x (y, z alike);  d2 = ((dx*dx) + (dy*dy)) + (dz*dz).
 * k_cap > 0 truncates a row to its k_cap smallest (d2, j); k_cap <= 0 keeps
 * the whole ball.  Rows are emitted in ascending j.
 *
 *   x_in [n_in, 3], x_out [n_out, 3]     device, float32
 *   in_splits, out_splits [n_batch + 1]  device, int32: cloud b owns inputs
 *                                        in_splits[b] .. in_splits[b+1]-1 and
 *                                        outputs out_splits[b] .. likewise;
 *                                        both start at 0 and end at n_in/n_out
 *   row_ptr [n_out + 1]                  device, output; row_ptr[n_out] = E
 *   col_idx [col_capacity]               device, output
 *   nnz_host                             host, may be NULL.  Non-NULL: E is
 *                                        read back (one stream synchronise);
 *                                        E > col_capacity returns
 *                                        SBC_ERR_CAPACITY with row_ptr filled
 *                                        and col_idx untouched; malformed
 *                                        splits return SBC_ERR_OUT_OF_RANGE.
 *                                        NULL: nothing is synchronised; writes
 *                                        past col_capacity are dropped, so the
 *                                        caller checks row_ptr[n_out] <=
 *                                        col_capacity before using col_idx.
 * ------------------------------------------------------------------------ */
/* Workspace of a point search with these sizes and this k_cap (a capped
 * search with 1 <= k_cap <= 512 visits the candidates once, into n_out rows of
 * k_cap entries held in the workspace). */
size_t sbc_points_workspace_size(int32_t n_in, int32_t n_out, int32_t n_batch, int32_t k_cap);
sbc_status sbc_neighbour_search_points(const float *x_in, int32_t n_in, const int32_t *in_splits,
                                       const float *x_out, int32_t n_out,
                                       const int32_t *out_splits, int32_t n_batch, float radius,
                                       int32_t k_cap, int32_t *row_ptr, int32_t *col_idx,
                                       int64_t col_capacity, int64_t *nnz_host, void *workspace,
                                       size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * 1b. Event neighbourhoods (Section 3.2: a small spatial block, extending
 * backwards in time only): event i's neighbours are the events j < i with
 * |px_i - px_j| <= half_extent, |py_i - py_j| <= half_extent and
 * t_i - t_j <= window.  A row lists them in block order: the block's pixels
 * row-major (dy, then dx, relative to event i's pixel), each pixel's events
 * in ascending j (the order a per-pixel search visits them).  The stream is
 * in place (outputs = inputs).
 *
 *   px, py, t [n]   device, int32; 0 <= px < width, 0 <= py < height, t
 *                   non-decreasing.  Events violating this never fault: they
 *                   are given no neighbours and, when nnz_host is non-NULL,
 *                   SBC_ERR_OUT_OF_RANGE / SBC_ERR_UNSORTED is returned.
 *   row_ptr, col_idx, col_capacity, nnz_host: as for points.
 * ------------------------------------------------------------------------ */
size_t sbc_events_workspace_size(int32_t n, int32_t width, int32_t height);
sbc_status sbc_neighbour_search_events(const int32_t *px, const int32_t *py, const int32_t *t,
                                       int32_t n, int32_t width, int32_t height,
                                       int32_t half_extent, int32_t window, int32_t *row_ptr,
                                       int32_t *col_idx, int64_t col_capacity, int64_t *nnz_host,
                                       void *workspace, size_t workspace_bytes,
                                       hipStream_t stream);

/* The same search, also emitting the transposed pattern (Section 3.1,
 * "Symmetry": the reverse neighbourhood), found from the same per-pixel lists
 * by the reverse search: column j lists the events i > j with |px_i - px_j|
 * <= half_extent, |py_i - py_j| <= half_extent and t_i - t_j <= window, in
 * block order around j (its block's pixels row-major relative to j's pixel,
 * ascending i within a pixel).  col_ptr [n + 1] equals what sbc_csr_transpose
 * gives for row_ptr / col_idx and row_idx holds the same entries per column,
 * in that order; no edge_perm is produced (see sbc_csc).  capacity bounds both col_idx and row_idx (E entries each);
 * the other arguments and the errors are those of sbc_neighbour_search_events,
 * whose workspace size it uses. */
sbc_status sbc_neighbour_search_events_csc(const int32_t *px, const int32_t *py,
                                           const int32_t *t, int32_t n, int32_t width,
                                           int32_t height, int32_t half_extent, int32_t window,
                                           int32_t *row_ptr, int32_t *col_idx, int32_t *col_ptr,
                                           int32_t *row_idx, int64_t capacity,
                                           int64_t *nnz_host, void *workspace,
                                           size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * 2. Basis values (Section 3.1, the values of the neighbourhood matrices):
 * v[e, m] = p_m(edge e) as float32, edge-major [E, M], in CSR edge order.
 * v must hold row_ptr[n_rows] * M floats.
 * ------------------------------------------------------------------------ */
sbc_status sbc_basis_eval(const sbc_csr *csr, const sbc_geometry *geometry, float *v,
                          hipStream_t stream);

/* ------------------------------------------------------------------------
 * 3. Transpose of the pattern, for the backward pass (Section 3.1,
 * "Symmetry": N_IJ = N_JI^T relates a neighbourhood to its reverse).
 * Stable: within a column, rows ascend.  col_ptr [n_cols + 1], row_idx and
 * edge_perm [E] are outputs.
 * ------------------------------------------------------------------------ */
size_t sbc_transpose_workspace_size(int32_t n_cols, int64_t nnz_bound);
sbc_status sbc_csr_transpose(const sbc_csr *csr, int32_t *col_ptr, int32_t *row_idx,
                             int32_t *edge_perm, void *workspace, size_t workspace_bytes,
                             hipStream_t stream);

/* The same transpose for a block-diagonal pattern: the CSR of a ragged batch
 * (Section 3.1, "Ragged Batching"), whose block b has the rows
 * row_splits[b] .. row_splits[b+1]-1 and the columns col_splits[b] ..
 * col_splits[b+1]-1 (for a point search: out_splits and in_splits).  Each
 * block is transposed on its own (one workgroup, in LDS), and the outputs
 * equal sbc_csr_transpose's.  No workspace.
 *   row_splits, col_splits [n_batch + 1]  device, int32, non-decreasing, from
 *                                         0 to n_rows and to n_cols
 * Entries whose column lies outside their block's columns are not transposed
 * (such a pattern is not block-diagonal: col_ptr then does not describe
 * them); every write stays inside col_ptr, row_idx and edge_perm. */
sbc_status sbc_csr_transpose_batched(const sbc_csr *csr, const int32_t *row_splits,
                                     const int32_t *col_splits, int32_t n_batch,
                                     int32_t *col_ptr, int32_t *row_idx, int32_t *edge_perm,
                                     hipStream_t stream);

/* ------------------------------------------------------------------------
 * 4. Forward: Y [n_out, C_out] float32 = sum_m N^(m) F W^(m) (Section 3.1,
 * the matrix-product form).
 *   v          [E, M] float32 basis values, or NULL to evaluate them inside the
 *              kernels from `geometry` (then geometry must be non-NULL)
 *   F          [n_in, C_in]      float32 or bf16 (dtype)
 *   W          [M, C_in, C_out]  float32 or bf16 (dtype)
 *   order      evaluation order (sbc_order)
 * ------------------------------------------------------------------------ */
/* Workspace of sbc_conv_forward and sbc_conv_backward (the larger of the two). */
size_t sbc_conv_workspace_size(int32_t n_out, int32_t n_in, int64_t nnz_bound, int32_t M,
                               int32_t C_in, int32_t C_out, sbc_dtype dtype, sbc_order order);
sbc_status sbc_conv_forward(const sbc_csr *csr, const float *v, const sbc_geometry *geometry,
                            int32_t M, const void *F, const void *W, sbc_dtype dtype,
                            int32_t C_in, int32_t C_out, float *Y, sbc_order order,
                            void *workspace, size_t workspace_bytes, hipStream_t stream);

/* The forward for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation):
 * sbc_conv_forward with the library's own static scratch in place of the
 * workspace.  The scratch is a device array of
 * sbc_conv_forward_noalloc_max_bytes() bytes (64 MiB) that each GPU the
 * library runs on holds until the process ends; the call itself allocates
 * nothing (no hipMalloc, no allocating library routine).  Arguments, results
 * and errors are those of sbc_conv_forward; a forward whose temporary space
 * (sbc_conv_workspace_size's forward share) exceeds the scratch returns
 * SBC_ERR_WORKSPACE and enqueues nothing.  No part of the scratch needs to
 * start at zero: every byte a call reads was written earlier in that call.
 * All calls on one GPU share its scratch, so calls that overlap on one GPU
 * (on different streams, or from different host threads without ordering)
 * race on it and must not be issued. */
size_t sbc_conv_forward_noalloc_max_bytes(void);
sbc_status sbc_conv_forward_noalloc(const sbc_csr *csr, const float *v,
                                    const sbc_geometry *geometry, int32_t M, const void *F,
                                    const void *W, sbc_dtype dtype, int32_t C_in, int32_t C_out,
                                    float *Y, sbc_order order, hipStream_t stream);

/* ------------------------------------------------------------------------
 * 5. Backward: the gradients of <Y, dY> with respect to F and W (Section 4,
 * Table 2: the backward pass of the matrix-product form, its gradients with
 * respect to the features and the kernel weights; as the forward, it can be
 * evaluated in either order of the products, Section 3.1 and Table 1).
 *   dY  [n_out, C_out]    float32 or bf16 (dtype)
 *   dF  [n_in, C_in]      float32 output, or NULL to skip
 *   dW  [M, C_in, C_out]  float32 output, or NULL to skip
 *   csc                   the transpose of csr (sbc_csr_transpose, or
 *                         sbc_neighbour_search_events_csc); its edge_perm
 *                         may be NULL only when v is NULL and the basis is
 *                         not SBC_BASIS_WMONO10
 * dW sums over every edge of the batch, in a fixed blocked order.
 * ------------------------------------------------------------------------ */
sbc_status sbc_conv_backward(const sbc_csr *csr, const sbc_csc *csc, const float *v,
                             const sbc_geometry *geometry, int32_t M, const void *F,
                             const void *W, const void *dY, sbc_dtype dtype, int32_t C_in,
                             int32_t C_out, float *dF, float *dW, sbc_order order,
                             void *workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * 5b. Gradient with respect to the decay rates of the learned-decay event
 * kernel (Section 3.2: lambda_uv is a learned parameter):
 *     dlambda[m] = d<Y, dY>/d lambda_m = sum_e v'[e, m] f_j W_m dy_i^T,
 * v' = d p_m / d lambda_m = -dt p_m.  dW' = sum_e v'[e, :] f_j^T dy_i is
 * formed like dW of the backward: with the transpose (csc non-NULL, its
 * edge_perm may be NULL) by the fused D-route where the shape has one, else
 * as G' = N' F (the sparse product with v') and dW' = G'^T dY; then
 * dlambda[m] = <dW'_m, W_m>.  Sums are taken in a fixed order.
 * geometry.basis must be SBC_BASIS_EVENT_DECAYS, M = 8 * n_decays.
 *   F [n, C_in], W [M, C_in, C_out], dY [n, C_out]  float32 or bf16 (dtype)
 *   dlambda [M]                                      float32 output
 * ------------------------------------------------------------------------ */
size_t sbc_decay_gradient_workspace_size(int32_t n, int64_t nnz_bound, int32_t M, int32_t C_in,
                                         int32_t C_out, sbc_dtype dtype);
sbc_status sbc_conv_decay_gradient(const sbc_csr *csr, const sbc_csc *csc,
                                   const sbc_geometry *geometry, int32_t M, const void *F,
                                   const void *W, const void *dY, sbc_dtype dtype, int32_t C_in,
                                   int32_t C_out, float *dlambda, void *workspace,
                                   size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * 6. The featureless convolution (Section 3.1, "Featureless Convolutions",
 * Eq. 9-10): every input carries the constant feature 1 (F = 1), so the
 * feature matrix drops out of the product,
 *     Z [n_out, P] = G~ Phi,   G~[i, m] = sum over row i of the values of p_m,
 * the first layer of a network on bare coordinates.
 *   v, geometry  the basis values [E, M], or NULL with the geometry (any basis)
 *   Phi          [M, P] float32 (the learned matrix Phi_0)
 *   Z            [n_out, P] float32 output
 * Row sums are taken in float64 in a fixed order.  The backward gives
 *   dPhi [M, P] = G~^T dZ   (float32; dZ [n_out, P] float32),
 * with the workspace of sbc_featureless_workspace_size (G~ and the split
 * partial sums of the contraction).  No pointer needs more than 4-byte
 * alignment.
 * ------------------------------------------------------------------------ */
size_t sbc_featureless_workspace_size(int32_t n_out, int32_t M, int32_t P);
sbc_status sbc_featureless_forward(const sbc_csr *csr, const float *v,
                                   const sbc_geometry *geometry, int32_t M, const float *Phi,
                                   int32_t P, float *Z, hipStream_t stream);
sbc_status sbc_featureless_backward(const sbc_csr *csr, const float *v,
                                    const sbc_geometry *geometry, int32_t M, const float *dZ,
                                    int32_t P, float *dPhi, void *workspace,
                                    size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * 7. Subsampling of a ragged point batch (Section 3.1, "Subsampling", and the
 * supplementary algorithms), cloud by cloud:
 *   SBC_SAMPLE_IFP                  iterative farthest points: repeatedly the
 *                                   point farthest from those taken (all
 *                                   distances start infinite, so the cloud's
 *                                   first point comes first);
 *   SBC_SAMPLE_APPROX_IFP           the same with each taken point lowering the
 *                                   distances of its ball neighbours only;
 *   SBC_SAMPLE_REJECTION            rejection sampling: in input order, every
 *                                   point that no earlier taken point has in
 *                                   its ball (a variable number per cloud);
 *   SBC_SAMPLE_APPROX_IFP_REJECTION rejection sampling, then the approximate
 *                                   farthest points from its distances up to
 *                                   per_cloud points (the taken points first,
 *                                   in input order; if rejection takes more,
 *                                   the first per_cloud of them).
 * Distances are compared as float32 squared distances in the canonical form of
 * the neighbour search; ties go to the lowest index, and the farthest-point
 * steps choose among the points not yet taken, so no point is output twice
 * (coincident points included).  Results are exact and deterministic.
 *   x [n_points, 3], splits [n_batch + 1]  device; clouds of at most max_cloud
 *                                          <= 8192 points (a larger cloud gets
 *                                          no outputs)
 *   ball        the in-place ball pattern of x (sbc_neighbour_search_points
 *               with x as inputs and outputs, k_cap <= 0); NULL for IFP
 *   per_cloud   outputs per cloud (min(per_cloud, cloud size)); ignored by
 *               SBC_SAMPLE_REJECTION
 *   out_idx     [n_points] device, output: global indices of the outputs,
 *               cloud by cloud, in the order taken
 *   out_splits  [n_batch + 1] device, output: cloud b's outputs are
 *               out_idx[out_splits[b] .. out_splits[b+1])
 *   dmin2       [n_points] device, output (may be NULL): each point's squared
 *               distance to its nearest taken point as the algorithm tracked it
 * ------------------------------------------------------------------------ */
typedef enum {
    SBC_SAMPLE_IFP = 0,
    SBC_SAMPLE_APPROX_IFP = 1,
    SBC_SAMPLE_REJECTION = 2,
    SBC_SAMPLE_APPROX_IFP_REJECTION = 3
} sbc_sampling;
size_t sbc_sampling_workspace_size(int32_t n_batch);
sbc_status sbc_sample_points(const float *x, const int32_t *splits, int32_t n_batch,
                             int32_t n_points, int32_t max_cloud, const sbc_csr *ball,
                             sbc_sampling method, int32_t per_cloud, int32_t *out_idx,
                             int32_t *out_splits, float *dmin2, void *workspace,
                             size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * 8. Event stream sampling by leaky integrate-and-fire (the supplementary's
 * algorithm for the coarser streams of the event networks, Section 4).
 *
 * The output grid has Wo = ceil(width / stride) x Ho = ceil(height / stride)
 * cells; cell (ox, oy) sees the kernel x kernel input pixels centred on
 * (ox * stride, oy * stride) (offsets -(kernel-1)/2 .. kernel/2, rounded down,
 * as in a padded strided convolution).  Every cell holds a potential V and the
 * time T of its last update, both 0 at the start.  For each input event i, in
 * stream order, every cell that sees its pixel (row-major over (oy, ox); n of
 * them) sets v = V * exp(-(t_i - T) / decay) + 1 / n; if v > v_thresh it emits
 * an output event (ox, oy, t_i) and sets v = v_reset; then V = v, T = t_i.
 * Potentials are float64, evaluated in that order with no fused multiply-add.
 * Output events come in emission order: by input event, then oy, then ox, so
 * their times are non-decreasing.  Deterministic.
 *   px, py, t   [n] int32 device: pixels in [0, width) x [0, height), times
 *               non-decreasing (an event off the sensor reaches no cell)
 *   kernel      1..5; stride >= 1 (with stride > kernel some pixels reach no
 *               cell, and their events change nothing)
 *   decay       the decay time (> 0; +inf: no decay); v_thresh, v_reset
 *   out_x, out_y, out_t  [capacity] int32 device, output: output events;
 *               out_src [capacity] (may be NULL): the input event that
 *               caused each.  At most n * ((kernel-1)/stride + 1)^2 events.
 *               Events past capacity are counted but not written.
 *   n_out_dev   int64 device (may be NULL): the number of output events
 *   n_out_host  (may be NULL) the same on the host; the call then synchronises
 *               the stream and reports SBC_ERR_OUT_OF_RANGE, SBC_ERR_UNSORTED
 *               or SBC_ERR_CAPACITY (without it, no synchronisation and no
 *               such checks, so the call can be captured in a graph)
 * ------------------------------------------------------------------------ */
size_t sbc_lif_workspace_size(int32_t n, int32_t width, int32_t height, int32_t kernel,
                              int32_t stride);
sbc_status sbc_lif_sample_events(const int32_t *px, const int32_t *py, const int32_t *t,
                                 int32_t n, int32_t width, int32_t height, int32_t kernel,
                                 int32_t stride, double decay, double v_thresh, double v_reset,
                                 int32_t *out_x, int32_t *out_y, int32_t *out_t,
                                 int32_t *out_src, int64_t capacity, int64_t *n_out_dev,
                                 int64_t *n_out_host, void *workspace, size_t workspace_bytes,
                                 hipStream_t stream);

/* ------------------------------------------------------------------------
 * 9. The event convolution's deployment form (Section 3.2, Eq. 13-15), for a
 * stream fed in batches, with the fixed decay of SBC_BASIS_EVENT8 (rate 1/tau
 * for every offset).
 *
 * The caller keeps the state: z [height * width, C_in] float32 and z_time
 * [height * width] int32, pixel y * width + x, both zero before the stream's
 * first batch (the paper's initial state).  For each event i of the batch, in
 * stream order, the output is read before the event's own update:
 *   Y[i] = sum over the 8 offsets u (the 3 x 3 block without its centre, basis
 *          index m(u) as in SBC_BASIS_EVENT8) of
 *          exp(-(t_i - z_time[q]) / tau) z[q] W[m(u)],  q = (px_i - ux, py_i - uy)
 *          on the sensor,
 * then z[x_i] = F[i] + exp(-(t_i - z_time[x_i]) / tau) z[x_i], z_time[x_i] = t_i.
 * The batch is computed in parallel with the recursion's value (decays of
 * earlier events in the batch compose with those of the state); sums and
 * decay factors are float64, z and Y float32.  Unlike the training form there
 * is no window: every earlier event counts, decayed.
 *   px, py, t  [n] int32 device: pixels on the sensor, times non-decreasing and
 *              not before the state's (not checked: no synchronisation; an
 *              event off the sensor reads its neighbours and updates no pixel)
 *   F          [n, C_in] float32 device; W [8, C_in, C_out] float32 device
 *   Y          [n, C_out] float32 device, output
 * The call never synchronises and allocates nothing, so a stream step can be
 * captured in a graph.
 * ------------------------------------------------------------------------ */
size_t sbc_event_stream_workspace_size(int32_t n, int32_t width, int32_t height, int32_t C_in,
                                       int32_t C_out);
sbc_status sbc_event_stream_step(const int32_t *px, const int32_t *py, const int32_t *t,
                                 const float *F, int32_t n, int32_t width, int32_t height,
                                 float tau, const float *W, int32_t C_in, int32_t C_out,
                                 float *z, int32_t *z_time, float *Y, void *workspace,
                                 size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * 10. The deployment form with learned decays (Section 3.2, Eq. 12-15): the
 * kernel of SBC_BASIS_EVENT_DECAYS, M_v = n_decays rates lambda_uv per offset
 * u, run as a recursion.  A pixel keeps one decayed sum per basis function
 * m = u * n_decays + v, since the functions of an offset decay at different
 * rates:
 *   Y[i] = sum over u, v of exp(-lambda_uv (t_i - z_time[q])) z[q, m] W[m],
 *          q = (px_i - ux, py_i - uy) on the sensor,
 * then z[x_i, m] = F[i] + exp(-lambda_uv (t_i - z_time[x_i])) z[x_i, m] for
 * every m, z_time[x_i] = t_i.  With every lambda_uv = 1/tau this is section 9
 * with W summed over v.
 *   decays     [8, n_decays] float32 device, the rates lambda_uv (> 0, not
 *              checked), 1 <= n_decays <= 4
 *   W          [8 * n_decays, C_in, C_out] float32 device
 *   z          [height * width, 8 * n_decays, C_in] float32 device, state;
 *              z_time [height * width] int32 device, state (both zero at the
 *              start, caller-owned)
 * Everything else, including the workspace, errors and synchronisation, is as
 * in section 9.  The workspace query returns 0 for invalid sizes.
 * ------------------------------------------------------------------------ */
size_t sbc_event_stream_decays_workspace_size(int32_t n, int32_t width, int32_t height,
                                              int32_t n_decays, int32_t C_in, int32_t C_out);
sbc_status sbc_event_stream_step_decays(const int32_t *px, const int32_t *py, const int32_t *t,
                                        const float *F, int32_t n, int32_t width, int32_t height,
                                        const float *decays, int32_t n_decays, const float *W,
                                        int32_t C_in, int32_t C_out, float *z, int32_t *z_time,
                                        float *Y, void *workspace, size_t workspace_bytes,
                                        hipStream_t stream);

/* ------------------------------------------------------------------------
 * Tracing, for measurement tools.  After sbc_trace_kernel(name, start, stop)
 * every launch of the kernel called `name` made by the calling thread records
 * `start` immediately before and `stop` immediately after itself on its
 * launch stream (a later launch re-records them).  NULL events remove the
 * entry, sbc_trace_clear() removes all entries.  sbc_kernel_names() lists the
 * traceable names, comma-separated.  Events stay owned by the caller.
 * ------------------------------------------------------------------------ */
sbc_status sbc_trace_kernel(const char *name, hipEvent_t start, hipEvent_t stop);
void sbc_trace_clear(void);
const char *sbc_kernel_names(void);

/*
 * The plan sbc_conv_forward / sbc_conv_backward follow for a shape.
 *   forward_order   SPMM_FIRST: (N F) W;  GEMM_FIRST: N (F W)
 *   backward_order  SPMM_FIRST: D = N^T dY first (dF = D Wt, dW = F^T D);
 *                   GEMM_FIRST: dG = dY W^T first (dF = N^T dG, dW = G^T dY)
 *   *_fused         1 when that pass runs as one fused kernel (gather into
 *                   LDS, basis evaluated inside, MFMA contraction), 0 when it
 *                   runs as separate gather and contraction kernels.
 * AUTO picks the order with the lower estimated cost: the multiply-adds of
 * the paper's cost table, plus 5e7 multiply-adds (about 5 us, measured) for
 * every kernel launch, a fused pass counting as two launches and a pass of
 * separate gather and contraction kernels as five.  The launch term only
 * matters for small problems, where it prefers the fused pass.  For the
 * backward the estimate is applied to the transposed problem.
 */
typedef struct {
    sbc_order forward_order;
    sbc_order backward_order;
    int32_t forward_fused;
    int32_t backward_fused;
} sbc_conv_plan_t;
sbc_status sbc_conv_plan(int32_t n_out, int32_t n_in, int64_t nnz_bound, int32_t M,
                         int32_t C_in, int32_t C_out, sbc_dtype dtype, sbc_order order,
                         sbc_conv_plan_t *plan);

/* The paper's rule alone: AUTO resolves to the order with fewer
 * multiply-adds (SBC_ORDER_SPMM_FIRST on a tie); an explicit order is returned
 * as given.  sbc_conv_plan adds the launch term above. */
sbc_order sbc_resolve_order(int32_t n_out, int32_t n_in, int64_t nnz, int32_t M, int32_t C_in,
                            int32_t C_out, sbc_order order);

#ifdef __cplusplus
}
#endif

#endif /* SBCONV_H */
