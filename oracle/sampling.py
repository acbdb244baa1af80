"""Subsampling of point clouds (Section 3.1, "Subsampling"; the supplementary
algorithms for iterative farthest point selection, its neighbourhood-limited
approximation and rejection sampling), in float32 where a comparison decides.

CPU ORACLE -- test infrastructure only (see the package docstring).

Distances are compared as squared float32 distances in the canonical form of
the neighbour search, d2 = ((dx*dx) + (dy*dy)) + (dz*dz) with dx = a.x - b.x
(the order of the square roots is the order of the squares).  Ties of the
farthest-point choice go to the lowest index.  Clouds are the ranges
splits[b] .. splits[b+1]-1 of a ragged batch; indices are global.
"""
from __future__ import annotations

import numpy as np


def _d2(x, j):
    """float32 squared distances from every point of x to x[j]."""
    d = x - x[j]
    return (d[:, 0] * d[:, 0] + d[:, 1] * d[:, 1]) + d[:, 2] * d[:, 2]


def ifp(x, splits, counts):
    """Iterative farthest points (the supplementary's first algorithm): start
    with every distance infinite, repeatedly take the point farthest from the
    points taken so far (argmax; the printed argmin is read as argmax, since
    with infinite initial distances argmin would take the first point again)
    and lower every distance to the new point.  The choice is among the points
    not yet taken (the farthest *remaining* point; it matters only once every
    remaining distance is 0, i.e. for coincident points).  Returns the global
    indices of each cloud's counts[b] points in the order taken, and the final
    squared distances [n]."""
    x = np.asarray(x, dtype=np.float32)
    out = []
    dall = np.full(len(x), np.inf, dtype=np.float32)
    for b in range(len(splits) - 1):
        s, e = int(splits[b]), int(splits[b + 1])
        xb = x[s:e]
        dmin = dall[s:e]
        taken = np.zeros(e - s, dtype=bool)
        for _ in range(int(counts[b])):
            j = int(np.argmax(np.where(taken, -1.0, dmin)))   # first index of the maximum
            taken[j] = True
            out.append(s + j)
            dmin[:] = np.minimum(dmin, _d2(xb, j))
    return np.asarray(out, dtype=np.int32), dall


def rejection_sampling(x, splits, row_ptr, col_idx):
    """Rejection sampling (the supplementary's fourth algorithm): visit the
    inputs in order; an input not yet visited is taken, and it and its ball
    neighbours (the in-place, uncapped neighbourhood CSR) are marked visited,
    each neighbour's distance lowered to its distance from the taken point.
    Returns (taken flags [n] int32, d_min squared [n] float32)."""
    x = np.asarray(x, dtype=np.float32)
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    col_idx = np.asarray(col_idx, dtype=np.int64)
    n = len(x)
    taken = np.zeros(n, dtype=np.int32)
    visited = np.zeros(n, dtype=bool)
    dmin = np.full(n, np.inf, dtype=np.float32)
    for i in range(n):
        if visited[i]:
            continue
        taken[i] = 1
        nb = col_idx[row_ptr[i]:row_ptr[i + 1]]
        visited[nb] = True
        d = x[nb] - x[i]
        d2 = (d[:, 0] * d[:, 0] + d[:, 1] * d[:, 1]) + d[:, 2] * d[:, 2]
        dmin[nb] = np.minimum(dmin[nb], d2)
    return taken, dmin


def approx_ifp(x, splits, counts, row_ptr, col_idx, dmin=None, taken=None):
    """Farthest points with distance updates limited to the ball neighbourhood
    of each taken point (the supplementary's approximate variant with a
    priority queue): take the remaining input of largest d_min (ties: lowest
    index; the queue gives up each input once, so a taken input is never
    taken again), then lower the d_min of its neighbours to their distance
    from it.  dmin: initial squared distances (rejection sampling's, for the
    variant that continues after it), else infinite; taken: inputs already
    taken (bool [n]), else none.  Returns the global indices taken, cloud by
    cloud, counts[b] per cloud, and the final squared distances."""
    x = np.asarray(x, dtype=np.float32)
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    col_idx = np.asarray(col_idx, dtype=np.int64)
    d = (np.full(len(x), np.inf, dtype=np.float32) if dmin is None
         else np.array(dmin, dtype=np.float32))
    done = np.zeros(len(x), dtype=bool) if taken is None else np.array(taken, dtype=bool)
    out = []
    for b in range(len(splits) - 1):
        s, e = int(splits[b]), int(splits[b + 1])
        for _ in range(int(counts[b])):
            j = s + int(np.argmax(np.where(done[s:e], -1.0, d[s:e])))
            done[j] = True
            out.append(j)
            nb = col_idx[row_ptr[j]:row_ptr[j + 1]]
            dd = x[nb] - x[j]
            d2 = (dd[:, 0] * dd[:, 0] + dd[:, 1] * dd[:, 1]) + dd[:, 2] * dd[:, 2]
            d[nb] = np.minimum(d[nb], d2)
    return np.asarray(out, dtype=np.int32), d


def approx_ifp_after_rejection(x, splits, per_cloud, row_ptr, col_idx):
    """Rejection sampling, then the approximate farthest points from its
    distances (the supplementary's last algorithm), per_cloud points per cloud
    (at most the cloud's size): the taken points first, in input order, then
    the farthest points.  When rejection takes more than per_cloud points the
    first per_cloud of them are kept (the output size is fixed; a reading, the
    algorithm leaves that case open).  Returns (indices, final squared distances)."""
    taken, d = rejection_sampling(x, splits, row_ptr, col_idx)
    out = []
    for b in range(len(splits) - 1):
        s, e = int(splits[b]), int(splits[b + 1])
        S = min(int(per_cloud), e - s)
        first = (s + np.nonzero(taken[s:e])[0])[:S]
        kept = np.zeros(len(x), dtype=bool)
        kept[first] = True
        more, d = approx_ifp(x, [s, e], [S - len(first)], row_ptr, col_idx, d, kept)
        out.extend(first.tolist())
        out.extend(more.tolist())
    return np.asarray(out, dtype=np.int32), d



def lif_receptive(x, kernel, stride, n_out):
    """Output cells (one dimension) whose receptive field holds input coordinate
    x.  Reading: cell o sees the kernel inputs centred on its own position o *
    stride, i.e. [o*stride - p, o*stride - p + kernel) with p = (kernel-1)//2,
    and there are ceil(size / stride) cells (a padded strided convolution, so
    each down-sampling halves the sensor as in the event networks)."""
    p = (kernel - 1) // 2
    return [o for o in range(n_out) if o * stride - p <= x < o * stride - p + kernel]


def lif(px, py, t, width, height, kernel, stride, decay, v_thresh, v_reset):
    """The leaky integrate-and-fire event sampler (the supplementary's
    algorithm for generating the next, coarser stream).  Every output cell
    keeps a potential V and the time T of its last update, both starting at 0.
    For each input event in stream order, each output cell of its receptive
    field N (row-major over (oy, ox)) decays its potential to the event's time,
    adds 1/n (n = |N|, the number of cells the event reaches), and, when the
    result exceeds v_thresh, resets it to v_reset and emits an output event at
    that cell with the input's time.  Potentials are float64.  Returns the
    (input event index, ox, oy) of every output event in emission order; the
    output grid has ceil(width / stride) x ceil(height / stride) cells."""
    Wo, Ho = -(-int(width) // stride), -(-int(height) // stride)
    V = np.zeros((Ho, Wo))
    T = np.zeros((Ho, Wo))
    out = []
    for i in range(len(t)):
        xs = lif_receptive(int(px[i]), kernel, stride, Wo)
        ys = lif_receptive(int(py[i]), kernel, stride, Ho)
        n = len(xs) * len(ys)
        ti = float(t[i])
        for oy in ys:
            for ox in xs:
                v = V[oy, ox] * np.exp(-(ti - T[oy, ox]) / decay) + 1.0 / n
                if v > v_thresh:
                    v = v_reset
                    out.append((i, ox, oy))
                V[oy, ox] = v
                T[oy, ox] = ti
    return np.asarray(out, dtype=np.int64).reshape(-1, 3)
