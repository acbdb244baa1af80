"""ctypes access to the oracle's C part (neighbour enumeration, transpose).

CPU ORACLE -- test infrastructure only: imported by the tests, the smoke check
and the benchmark's CPU-baseline leg, never by the product package.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "neighbours.c")
LIB_PATH = os.path.join(_HERE, "liboracle.so")

_i32p = ctypes.POINTER(ctypes.c_int32)
_f32p = ctypes.POINTER(ctypes.c_float)


def build(force: bool = False) -> str:
    """Compile the C part with gcc (no fp contraction, OpenMP over rows)."""
    if force or not os.path.exists(LIB_PATH) or os.path.getmtime(LIB_PATH) < os.path.getmtime(_SRC):
        tmp = LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c99", "-ffp-contract=off", "-fopenmp",
                               "-shared", "-fPIC", "-o", tmp, _SRC])
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


_lib = None


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(LIB_PATH)
        L.orc_points_brute.restype = ctypes.c_int64
        L.orc_points_brute.argtypes = [_f32p, _i32p, _f32p, _i32p, ctypes.c_int32, ctypes.c_int32,
                                       ctypes.c_float, ctypes.c_int32, _i32p, _i32p]
        L.orc_points_d2.restype = ctypes.c_int64
        L.orc_points_d2.argtypes = [_f32p, _f32p, _i32p, _i32p, ctypes.c_int32, _f32p]
        for name in ("orc_events_quadratic", "orc_events_scan"):
            f = getattr(L, name)
            f.restype = ctypes.c_int64
            f.argtypes = [_i32p, _i32p, _i32p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                          _i32p, _i32p]
        L.orc_events_pixels.restype = ctypes.c_int64
        L.orc_events_pixels.argtypes = [_i32p, _i32p, _i32p, ctypes.c_int32, ctypes.c_int32,
                                        ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                        _i32p, _i32p]
        L.orc_csr_transpose.restype = None
        L.orc_csr_transpose.argtypes = [_i32p, _i32p, ctypes.c_int32, ctypes.c_int32,
                                        _i32p, _i32p, _i32p]
        L.orc_max_threads.restype = ctypes.c_int
        _lib = L
    return _lib


def _p(a, t):
    return a.ctypes.data_as(t)


def max_threads() -> int:
    return int(lib().orc_max_threads())


def points_csr(x_in, in_splits, x_out, out_splits, radius, k_cap):
    """CSR of the (capped) ball neighbourhoods of a ragged point batch."""
    x_in = np.ascontiguousarray(x_in, dtype=np.float32)
    x_out = np.ascontiguousarray(x_out, dtype=np.float32)
    in_splits = np.ascontiguousarray(in_splits, dtype=np.int32)
    out_splits = np.ascontiguousarray(out_splits, dtype=np.int32)
    n_out = len(x_out)
    n_batch = len(out_splits) - 1
    row_ptr = np.zeros(n_out + 1, dtype=np.int32)
    args = (_p(x_in, _f32p), _p(in_splits, _i32p), _p(x_out, _f32p), _p(out_splits, _i32p),
            n_batch, n_out, ctypes.c_float(np.float32(radius)), int(k_cap))
    E = lib().orc_points_brute(*args, _p(row_ptr, _i32p), None)
    col_idx = np.zeros(max(E, 1), dtype=np.int32)
    lib().orc_points_brute(*args, _p(row_ptr, _i32p), _p(col_idx, _i32p))
    return row_ptr, col_idx[:E]


def points_d2(x_in, x_out, row_ptr, col_idx):
    """fp32 squared distance of each edge, evaluated as in the neighbour test."""
    x_in = np.ascontiguousarray(x_in, dtype=np.float32)
    x_out = np.ascontiguousarray(x_out, dtype=np.float32)
    row_ptr = np.ascontiguousarray(row_ptr, dtype=np.int32)
    col_idx = np.ascontiguousarray(col_idx, dtype=np.int32)
    d2 = np.zeros(max(len(col_idx), 1), dtype=np.float32)
    lib().orc_points_d2(_p(x_in, _f32p), _p(x_out, _f32p), _p(row_ptr, _i32p),
                        _p(col_idx, _i32p), len(row_ptr) - 1, _p(d2, _f32p))
    return d2[:len(col_idx)]


def block_order(ptr, idx, px, py, half_extent):
    """Entries of each segment r (ptr[r] .. ptr[r+1]) of an event pattern, the
    events near event r, ordered by the position of their pixel in r's block,
    row-major over (dy, dx) relative to r's pixel, then by index (stream
    order within a pixel)."""
    ptr = np.asarray(ptr, dtype=np.int64)
    idx = np.asarray(idx, dtype=np.int32)
    px = np.asarray(px, dtype=np.int64)
    py = np.asarray(py, dtype=np.int64)
    h = int(half_extent)
    seg = np.repeat(np.arange(len(ptr) - 1), np.diff(ptr))
    pos = (py[idx] - py[seg] + h) * (2 * h + 1) + (px[idx] - px[seg] + h)
    return idx[np.lexsort((idx, pos, seg))].astype(np.int32)


def events_csr(px, py, t, window, half_extent=1, width=None, height=None, method="pixels"):
    """CSR of the backwards-in-time pixel-block neighbourhoods of an event stream.
    A row lists the block's pixels in row-major order, each pixel's events in
    stream order (block_order): the order a per-pixel search visits them.

    method: 'pixels' (per-pixel lists), 'scan' (every event of the time window
    tested) or 'quadratic' (every earlier event tested); each finds a row's
    events in stream order, then the row is put in block order.
    """
    px = np.ascontiguousarray(px, dtype=np.int32)
    py = np.ascontiguousarray(py, dtype=np.int32)
    t = np.ascontiguousarray(t, dtype=np.int32)
    n = len(t)
    if n > 1 and np.any(np.diff(t.astype(np.int64)) < 0):
        raise ValueError("timestamps must be non-decreasing")
    row_ptr = np.zeros(n + 1, dtype=np.int32)
    if method == "pixels":
        if width is None:
            width = int(px.max()) + 1 if n else 1
        if height is None:
            height = int(py.max()) + 1 if n else 1
        f = lambda rp, ci: lib().orc_events_pixels(_p(px, _i32p), _p(py, _i32p), _p(t, _i32p), n,
                                                   int(width), int(height), int(half_extent),
                                                   int(window), rp, ci)
    else:
        fn = {"scan": lib().orc_events_scan, "quadratic": lib().orc_events_quadratic}[method]
        f = lambda rp, ci: fn(_p(px, _i32p), _p(py, _i32p), _p(t, _i32p), n, int(half_extent),
                              int(window), rp, ci)
    E = f(_p(row_ptr, _i32p), None)
    col_idx = np.zeros(max(E, 1), dtype=np.int32)
    f(_p(row_ptr, _i32p), _p(col_idx, _i32p))
    return row_ptr, block_order(row_ptr, col_idx[:E], px, py, half_extent)


def events_csc(px, py, t, window, half_extent=1, width=None, height=None, method="pixels"):
    """The transposed event pattern (the reverse neighbourhoods): column j
    lists the events i > j whose block holds j's pixel and t_i - t_j <=
    window, in block order around j (block_order with j as the centre).
    Returns (col_ptr, row_idx)."""
    rp, ci = events_csr(px, py, t, window, half_extent, width, height, method)
    cp, ri, _ = csr_transpose(rp, ci, len(np.asarray(t)))
    return cp, block_order(cp, ri, px, py, half_extent)


def csr_transpose(row_ptr, col_idx, n_cols):
    """Stable transpose: (col_ptr, row_idx, edge_perm), rows ascending in each column."""
    row_ptr = np.ascontiguousarray(row_ptr, dtype=np.int32)
    col_idx = np.ascontiguousarray(col_idx, dtype=np.int32)
    E = len(col_idx)
    col_ptr = np.zeros(n_cols + 1, dtype=np.int32)
    row_idx = np.zeros(max(E, 1), dtype=np.int32)
    perm = np.zeros(max(E, 1), dtype=np.int32)
    lib().orc_csr_transpose(_p(row_ptr, _i32p), _p(col_idx, _i32p), len(row_ptr) - 1, n_cols,
                            _p(col_ptr, _i32p), _p(row_idx, _i32p), _p(perm, _i32p))
    return col_ptr, row_idx[:E], perm[:E]
