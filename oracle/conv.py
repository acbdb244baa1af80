"""The sparse basis convolution and its gradients, by definition, in float64.

CPU ORACLE -- test infrastructure only (see the package docstring).

Forward (Section 3.1, the finite convolution sum with the kernel written as a
linear combination of basis functions): for every output i,

    y_i = sum_{j in N_i} f_j g(dx_ij),     g(dx) = sum_m p_m(dx) W_m,

with f_j the C_in features of input j (a row vector), W_m a C_in x C_out
matrix and p_m(dx_ij) the basis value v[e, m] of edge e = (i, j).  This is the
plain definition; the method's reordering into sum_m (N_m F) W_m is *not*
used here.

Backward: the exact derivatives of the scalar <Y, dY> with respect to the
features and the weights of that same sum, per edge:

    dW_m += v[e, m] * f_j^T dy_i,        df_j += g(dx_ij) dy_i^T.

Everything is evaluated in float64 on the exact input values (bf16 inputs are
passed as the float32 numbers they denote).
"""
from __future__ import annotations

import numpy as np

from .basis import edge_rows

_CHUNK_DOUBLES = 1 << 24    # bound on the per-chunk kernel tensor


def _edge_chunks(edges, per_edge):
    step = max(1, _CHUNK_DOUBLES // max(1, per_edge))
    for s in range(0, len(edges), step):
        yield edges[s:s + step]


def _edge_kernels(v_e, Wd):
    """g(dx_e) = sum_m v[e, m] W_m for a block of edges: [n_e, C_in, C_out]."""
    M, cin, cout = Wd.shape
    return (v_e @ Wd.reshape(M, cin * cout)).reshape(len(v_e), cin, cout)


def forward(row_ptr, col_idx, v, F, W, rows=None):
    """Y[rows] (all rows when rows is None): y_i = sum_e f_j g(dx_e)."""
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    cols = np.asarray(col_idx, dtype=np.int64)
    Fd = np.asarray(F, dtype=np.float64)
    Wd = np.asarray(W, dtype=np.float64)
    vd = np.asarray(v, dtype=np.float64)
    M, cin, cout = Wd.shape
    n_out = len(row_ptr) - 1
    rows = np.arange(n_out) if rows is None else np.asarray(rows, dtype=np.int64)
    Y = np.zeros((len(rows), cout))
    lens = row_ptr[rows + 1] - row_ptr[rows]
    edges = (np.repeat(row_ptr[rows] - np.cumsum(lens) + lens, lens)
             + np.arange(int(lens.sum())))
    local = np.repeat(np.arange(len(rows)), lens)
    for pos in _edge_chunks(np.arange(len(edges)), cin * cout):
        e = edges[pos]
        K = _edge_kernels(vd[e], Wd)
        contrib = np.matmul(Fd[cols[e]][:, None, :], K)[:, 0, :]
        np.add.at(Y, local[pos], contrib)
    return Y


def backward(row_ptr, col_idx, v, F, W, dY, n_in, cols_subset=None, want_dW=True):
    """(dF, dW): dF for all inputs (or only the rows `cols_subset`), dW [M, C_in, C_out]."""
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    cols = np.asarray(col_idx, dtype=np.int64)
    Fd = np.asarray(F, dtype=np.float64)
    Wd = np.asarray(W, dtype=np.float64)
    vd = np.asarray(v, dtype=np.float64)
    dYd = np.asarray(dY, dtype=np.float64)
    M, cin, cout = Wd.shape
    rows = edge_rows(row_ptr)

    dW = None
    if want_dW:
        dW = np.zeros((M, cin, cout))
        for e in _edge_chunks(np.arange(len(cols)), cin * M):
            Fe = Fd[cols[e]]
            Ye = dYd[rows[e]]
            for m in range(M):
                dW[m] += (Fe * vd[e, m:m + 1]).T @ Ye

    if cols_subset is None:
        sel = np.arange(len(cols))
        target = np.arange(n_in)
    else:
        target = np.asarray(cols_subset, dtype=np.int64)
        sel = np.nonzero(np.isin(cols, target))[0]
    pos_of = np.full(n_in, -1, dtype=np.int64)
    pos_of[target] = np.arange(len(target))
    dF = np.zeros((len(target), cin))
    for e in _edge_chunks(sel, cin * cout):
        K = _edge_kernels(vd[e], Wd)
        contrib = np.matmul(K, dYd[rows[e]][:, :, None])[:, :, 0]
        np.add.at(dF, pos_of[cols[e]], contrib)
    return dF, dW


def featureless_forward(row_ptr, col_idx, v, Phi):
    """The featureless convolution (Section 3.1, "Featureless Convolutions",
    Eq. 9-10): every input carries the constant feature 1 (F = 1), so Z =
    G~ Phi_0, where G~[i, m] adds up the values of basis function m along row i
    and Phi_0 is an M x P matrix (P output channels).  Returns (Z [n_out, P],
    G~ [n_out, M])."""
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    vd = np.asarray(v, dtype=np.float64)
    n_out = len(row_ptr) - 1
    Gt = np.zeros((n_out, vd.shape[1]))
    rows = edge_rows(row_ptr)
    np.add.at(Gt, rows, vd)
    return Gt @ np.asarray(Phi, dtype=np.float64), Gt


def featureless_backward(row_ptr, col_idx, v, dZ):
    """Gradient of <Z, dZ> with respect to Phi_0: G~^T dZ (M x P)."""
    _, Gt = featureless_forward(row_ptr, col_idx, v, np.zeros((np.asarray(v).shape[1], 1)))
    return Gt.T @ np.asarray(dZ, dtype=np.float64)


def decay_backward(row_ptr, col_idx, v_deriv, F, W, dY):
    """Gradient of <Y, dY> with respect to the decay rates of the event kernel
    (Section 3.2, Eq. 12: lambda_uv is learned), by the chain rule per edge:
    d<Y, dY>/d lambda_m = sum_e v'[e, m] f_j W_m dy_i^T, with v' the values of
    d p_m / d lambda_m (oracle.basis.event_decay_basis(..., derivative=True))."""
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    rows = edge_rows(row_ptr)
    cols = np.asarray(col_idx, dtype=np.int64)
    Fd = np.asarray(F, dtype=np.float64)
    Wd = np.asarray(W, dtype=np.float64)
    dYd = np.asarray(dY, dtype=np.float64)
    vd = np.asarray(v_deriv, dtype=np.float64)
    M = Wd.shape[0]
    out = np.zeros(M)
    for m in range(M):
        nz = np.nonzero(vd[:, m])[0]
        if len(nz) == 0:
            continue
        fw = Fd[cols[nz]] @ Wd[m]                      # [n_e, C_out]
        out[m] = np.sum(vd[nz, m] * np.einsum("ij,ij->i", fw, dYd[rows[nz]]))
    return out


def deployment_stream(px, py, t, F, W, width, height, tau, z=None, last=None, decays=None):
    """The event convolution's deployment form (Section 3.2, Eq. 13-15): each
    pixel x keeps, for every basis function (u, v), z_x^(uv), the sum of the
    features of its events decayed at rate lambda_uv, and tau_x, the time of
    its last update (all 0 at the start).  An event (x, t) with features f
    first reads its output, the sum over the 8 offsets u and the decays v of
    exp(-lambda_uv (t - tau_q)) z_q^(uv) W_(u,v) with q = x - u on the sensor
    (the centre has no function), then updates its own pixel:
    z_x^(uv) <- f + exp(-lambda_uv (t - tau_x)) z_x^(uv), tau_x <- t.
    Events in stream order, float64.

    decays None: one rate 1/tau for every function (M_v = 1); every z^(u) of a
    pixel is then the same, so one is kept, z [H, W, C_in], and W is
    [8, C_in, C_out].  decays [8, M_v]: lambda_uv, z [H, W, 8, M_v, C_in] and W
    [8 M_v, C_in, C_out] with function m = u M_v + v.  z and last carry the
    state between calls (a stream fed in pieces); returns (Y, z, last)."""
    from .basis import event_offset_index
    C_in, C_out = W.shape[1], W.shape[2]
    lam = (np.full((8, 1), 1.0 / tau) if decays is None
           else np.asarray(decays, dtype=np.float64))
    Mv = lam.shape[1]
    shape = (height, width, C_in) if decays is None else (height, width, 8, Mv, C_in)
    z = np.zeros(shape) if z is None else np.array(z, dtype=np.float64)
    last = np.zeros((height, width)) if last is None else np.array(last, dtype=np.float64)
    state = (lambda y, x, u, v: z[y, x]) if decays is None else \
        (lambda y, x, u, v: z[y, x, u, v])
    Y = np.zeros((len(t), C_out))
    for i in range(len(t)):
        x, y, ti = int(px[i]), int(py[i]), float(t[i])
        for uy in (-1, 0, 1):
            for ux in (-1, 0, 1):
                u = int(event_offset_index(ux, uy))
                qx, qy = x - ux, y - uy
                if u < 0 or not (0 <= qx < width and 0 <= qy < height):
                    continue
                for v in range(Mv):
                    Y[i] += (np.exp(-lam[u, v] * (ti - last[qy, qx])) * state(qy, qx, u, v)
                             @ W[u * Mv + v])
        if decays is None:
            z[y, x] = F[i] + np.exp(-lam[0, 0] * (ti - last[y, x])) * z[y, x]
        else:
            for u in range(8):
                for v in range(Mv):
                    z[y, x, u, v] = F[i] + np.exp(-lam[u, v] * (ti - last[y, x])) * z[y, x, u, v]
        last[y, x] = ti
    return Y, z, last
