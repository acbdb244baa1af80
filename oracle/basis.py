"""Basis values of the neighbourhood matrices, in float64.

CPU ORACLE -- test infrastructure only (see the package docstring).

The values n_ij^(m) of the M sparse matrices (Section 3.1, the entries of the
neighbourhood matrices: the m-th basis function at the edge vector
dx_ij = x'_i - x_j, zero off the neighbourhood) are computed per edge, in the
CSR order of the edges.
"""
from __future__ import annotations

import numpy as np


def edge_rows(row_ptr):
    """Row (output) index of every edge of a CSR."""
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    return np.repeat(np.arange(len(row_ptr) - 1), np.diff(row_ptr))


def point_basis(x_in, x_out, row_ptr, col_idx, radius, M):
    """Monomials of u = (x'_i - x_j) / r times the window w = (1 - |u|^2)^2.

    Section 3.1 uses geometric monomials of the edge vector as the fixed basis
    (the kernel as a linear combination of unlearned basis functions).  The
    order is M = 4: [1, ux, uy, uz];  M = 8: [1, ux, uy, uz, ux^2, uy^2, uz^2,
    ux*uy], each multiplied by w.  r is taken as the float32 radius the search
    used; the coordinate differences are exact in float64.
    """
    r = float(np.float32(radius))
    rows = edge_rows(row_ptr)
    cols = np.asarray(col_idx, dtype=np.int64)
    u = (np.asarray(x_out, np.float64)[rows] - np.asarray(x_in, np.float64)[cols]) / r
    ux, uy, uz = u[:, 0], u[:, 1], u[:, 2]
    s = ux * ux + uy * uy + uz * uz
    w = (1.0 - s) ** 2
    one = np.ones_like(ux)
    if M == 4:
        mono = [one, ux, uy, uz]
    elif M == 8:
        mono = [one, ux, uy, uz, ux * ux, uy * uy, uz * uz, ux * uy]
    else:
        raise ValueError("point basis supports M = 4 or M = 8")
    return np.stack([m * w for m in mono], axis=1)


def weighted_point_basis(x_in, x_out, row_ptr, col_idx, radius):
    """The weighted convolution's values with the full second-order monomials.

    Section 3.1, "Weighted Convolutions" (Eq. 11): every value of row i is
    multiplied by w_ij / W_i, with w_ij = 1 - |dx_ij| / r, which falls to zero
    at the ball radius, and W_i the sum of w_ij over the row.  The basis is
    the full set of monomials up to second order of u = dx / r that the
    paper's networks use (M = 10): [1, ux, uy, uz, ux^2, uy^2, uz^2, ux*uy,
    ux*uz, uy*uz], with no other window.  A row whose weights sum to zero gets
    zero values.  r is the float32 radius of the search; coordinate
    differences are exact in float64.
    """
    r = float(np.float32(radius))
    rows = edge_rows(row_ptr)
    cols = np.asarray(col_idx, dtype=np.int64)
    d = np.asarray(x_out, np.float64)[rows] - np.asarray(x_in, np.float64)[cols]
    u = d / r
    ux, uy, uz = u[:, 0], u[:, 1], u[:, 2]
    w = 1.0 - np.sqrt((d * d).sum(axis=1)) / r
    n_rows = len(row_ptr) - 1
    W = np.zeros(n_rows, dtype=np.float64)
    np.add.at(W, rows, w)
    Wr = W[rows]
    scale = np.divide(w, Wr, out=np.zeros_like(w), where=Wr != 0.0)
    mono = [np.ones_like(ux), ux, uy, uz, ux * ux, uy * uy, uz * uz, ux * uy, ux * uz, uy * uz]
    return np.stack([m * scale for m in mono], axis=1)


def point_values(basis, x_in, x_out, row_ptr, col_idx, radius, M):
    """Values of a point basis by name: "wmono10" is the weighted convolution,
    any other name the windowed monomials of M functions."""
    if basis == "wmono10":
        return weighted_point_basis(x_in, x_out, row_ptr, col_idx, radius)
    return point_basis(x_in, x_out, row_ptr, col_idx, radius, M)


def event_offset_index(ux, uy, half_extent=1):
    """Basis index of pixel offset (ux, uy): row-major over (uy, ux), centre removed.

    Returns -1 for the centre offset, which has no basis function.
    """
    side = 2 * half_extent + 1
    k = (np.asarray(uy) + half_extent) * side + (np.asarray(ux) + half_extent)
    centre = half_extent * side + half_extent
    return np.where(k == centre, -1, np.where(k < centre, k, k - 1))


def event_basis(px, py, t, row_ptr, col_idx, tau, half_extent=1):
    """One-hot pixel-offset basis times exp(-dt / tau) (Section 3.2).

    The event kernel is a sum over spatial offsets u of exp(-lambda dt) theta_u;
    with one decay per offset (lambda = 1/tau) this is M = (2h+1)^2 - 1 basis
    functions (the centre offset dropped), each the indicator of one offset
    times the decay.  u = (px_i - px_j, py_i - py_j), dt = t_i - t_j >= 0.
    Edges between events of the same pixel have an all-zero basis row.
    """
    rows = edge_rows(row_ptr)
    cols = np.asarray(col_idx, dtype=np.int64)
    px = np.asarray(px, dtype=np.int64)
    py = np.asarray(py, dtype=np.int64)
    t = np.asarray(t, dtype=np.int64)
    ux = px[rows] - px[cols]
    uy = py[rows] - py[cols]
    dt = (t[rows] - t[cols]).astype(np.float64)
    m = event_offset_index(ux, uy, half_extent)
    M = (2 * half_extent + 1) ** 2 - 1
    v = np.zeros((len(cols), M), dtype=np.float64)
    hit = m >= 0
    v[np.nonzero(hit)[0], m[hit]] = np.exp(-dt[hit] / float(tau))
    return v


def event_values(basis, px, py, t, row_ptr, col_idx, tau, decays=None):
    """Values of an event basis by name: "event_decays" is the learned-decay
    kernel with the rates `decays` [8, M_v], any other name the fixed decay 1/tau."""
    if basis == "event_decays":
        return event_decay_basis(px, py, t, row_ptr, col_idx, decays)
    return event_basis(px, py, t, row_ptr, col_idx, tau)


def event_decay_basis(px, py, t, row_ptr, col_idx, lam, half_extent=1, derivative=False):
    """The event kernel with several learned decays per offset (Section 3.2,
    Eq. 12): g(u, dt) = sum_v exp(-lambda_uv dt) theta_uv, i.e. the basis
    functions p_uv = [offset == u] exp(-lambda_uv dt), M = M_u M_v of them,
    numbered m = u M_v + v (u the offset index with the centre removed).
    lam: [M_u, M_v] decay rates.  derivative: the values of d p_uv / d lambda_uv
    = -dt p_uv instead (the basis of the decay gradient).
    """
    lam = np.asarray(lam, dtype=np.float64)
    Mu, Mv = lam.shape
    rows = edge_rows(row_ptr)
    cols = np.asarray(col_idx, dtype=np.int64)
    px = np.asarray(px, dtype=np.int64)
    py = np.asarray(py, dtype=np.int64)
    t = np.asarray(t, dtype=np.int64)
    u = event_offset_index(px[rows] - px[cols], py[rows] - py[cols], half_extent)
    dt = (t[rows] - t[cols]).astype(np.float64)
    v = np.zeros((len(cols), Mu * Mv), dtype=np.float64)
    hit = np.nonzero(u >= 0)[0]
    for q in range(Mv):
        val = np.exp(-lam[u[hit], q] * dt[hit])
        if derivative:
            val = -dt[hit] * val
        v[hit, u[hit] * Mv + q] = val
    return v
