"""Python binding of the sbconv C ABI on torch tensors.

Argument marshalling only: every step runs in the HIP library.  torch supplies
device memory (outputs and workspaces) and the current HIP stream.  Inputs
must already be contiguous device tensors of the documented dtypes; nothing is
converted or moved implicitly.
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass
from typing import Optional, Tuple

import torch

from . import _lib as L

ORDERS = {"auto": L.SBC_ORDER_AUTO, "spmm_first": L.SBC_ORDER_SPMM_FIRST,
          "gemm_first": L.SBC_ORDER_GEMM_FIRST}
BASES = {"mono4": L.SBC_BASIS_MONO4, "mono8": L.SBC_BASIS_MONO8, "event8": L.SBC_BASIS_EVENT8,
         "wmono10": L.SBC_BASIS_WMONO10, "event_decays": L.SBC_BASIS_EVENT_DECAYS}
BASIS_M = {"mono4": 4, "mono8": 8, "event8": 8, "wmono10": 10}


def _require(t: torch.Tensor, name: str, dtype, ndim=None, device=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device (cuda/HIP) tensor, got {t.device}")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if dtype is not None and t.dtype not in (dtype if isinstance(dtype, tuple) else (dtype,)):
        raise ValueError(f"{name} must have dtype {dtype}, got {t.dtype}")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must be {ndim}-D, got shape {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _p(t: Optional[torch.Tensor]):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


class _Workspace:
    """A 256-byte aligned device buffer of at least `nbytes`."""

    def __init__(self, nbytes: int, device):
        self.buf = torch.empty(int(nbytes) + 256, dtype=torch.uint8, device=device)
        base = self.buf.data_ptr()
        self.ptr = ctypes.c_void_p(base + (-base) % 256)
        self.nbytes = int(nbytes)


@dataclass
class CSR:
    """Neighbourhood pattern: rows are outputs, columns inputs."""
    row_ptr: torch.Tensor      # int32 [n_rows + 1]
    col_idx: torch.Tensor      # int32 [>= nnz]
    n_rows: int
    n_cols: int
    nnz: int                   # exact edge count (or an upper bound when not synchronised)

    def c_struct(self) -> L.SbcCsr:
        return L.SbcCsr(self.n_rows, self.n_cols, self.nnz, self.row_ptr.data_ptr(),
                        self.col_idx.data_ptr())


@dataclass
class CSC:
    """Transposed pattern: rows are inputs.  edge_perm (each entry's CSR
    position) may be None when the basis is evaluated inside the kernels."""
    col_ptr: torch.Tensor               # int32 [n_cols + 1]
    row_idx: torch.Tensor               # int32 [nnz]
    edge_perm: Optional[torch.Tensor]   # int32 [nnz] or None
    n_cols: int

    def c_struct(self) -> L.SbcCsc:
        perm = self.edge_perm.data_ptr() if self.edge_perm is not None else None
        return L.SbcCsc(self.n_cols, self.col_ptr.data_ptr(), self.row_idx.data_ptr(), perm)


@dataclass
class Geometry:
    """Coordinates the basis is evaluated from (points: x_in/x_out/radius; events:
    px/py/t and tau, or for "event_decays" the rates `decays` [8, n_decays])."""
    basis: str
    radius: float = 0.0
    tau: float = 0.0
    x_in: Optional[torch.Tensor] = None
    x_out: Optional[torch.Tensor] = None
    px: Optional[torch.Tensor] = None
    py: Optional[torch.Tensor] = None
    t: Optional[torch.Tensor] = None
    decays: Optional[torch.Tensor] = None

    @property
    def M(self) -> int:
        if self.basis == "event_decays":
            return 8 * int(self.decays.shape[1])
        return BASIS_M[self.basis]

    def check(self, csr: "CSR") -> None:
        """Dtype, device, contiguity and length of every coordinate tensor the
        basis reads, against the pattern's sizes (the kernels index them by
        the pattern's rows and columns)."""
        if self.basis not in BASES:
            raise ValueError(f"unknown basis {self.basis!r}")
        dev = csr.row_ptr.device
        if self.basis in ("mono4", "mono8", "wmono10"):
            for name, x, n in (("x_in", self.x_in, csr.n_cols), ("x_out", self.x_out, csr.n_rows)):
                if x is None:
                    raise ValueError(f"geometry.{name} is needed for the point basis")
                _require(x, name, torch.float32, 2, dev)
                if tuple(x.shape) != (n, 3):
                    raise ValueError(f"{name} must be [{n}, 3], got {tuple(x.shape)}")
            return
        n = max(csr.n_rows, csr.n_cols)     # an event stream is in place
        for name, x in (("px", self.px), ("py", self.py), ("t", self.t)):
            if x is None:
                raise ValueError(f"geometry.{name} is needed for the event basis")
            _require(x, name, torch.int32, 1, dev)
            if x.numel() != n:
                raise ValueError(f"{name} must hold {n} events, got {x.numel()}")
        if self.basis == "event_decays":
            if self.decays is None:
                raise ValueError("geometry.decays is needed for the learned-decay basis")
            _require(self.decays, "decays", torch.float32, 2, dev)
            if self.decays.shape[0] != 8 or not 2 <= self.decays.shape[1] <= 4:
                raise ValueError("decays must be [8, n_decays] with 2 <= n_decays <= 4")

    def c_struct(self) -> L.SbcGeometry:
        d = lambda x: x.data_ptr() if x is not None else 0
        nd = int(self.decays.shape[1]) if self.decays is not None else 0
        if self.decays is not None:
            _require(self.decays, "decays", torch.float32, 2)
        return L.SbcGeometry(BASES[self.basis], float(self.radius), float(self.tau), d(self.x_in),
                             d(self.x_out), d(self.px), d(self.py), d(self.t), d(self.decays), nd)


def neighbour_search_points(x_in, in_splits, x_out, out_splits, radius: float, k_cap: int,
                            col_capacity: Optional[int] = None, sync: bool = True) -> CSR:
    """Ball (k-capped) neighbourhoods of a ragged point batch -> CSR (sbc_neighbour_search_points).

    sync=True reads E back (exact CSR, errors reported); sync=False never
    synchronises and requires k_cap > 0 (the capacity is n_out * k_cap).
    """
    _require(x_in, "x_in", torch.float32, 2)
    dev = x_in.device
    _require(x_out, "x_out", torch.float32, 2, dev)
    _require(in_splits, "in_splits", torch.int32, 1, dev)
    _require(out_splits, "out_splits", torch.int32, 1, dev)
    n_in, n_out = x_in.shape[0], x_out.shape[0]
    n_batch = in_splits.numel() - 1
    if out_splits.numel() != n_batch + 1:
        raise ValueError("in_splits and out_splits must have the same length")
    if col_capacity is None:
        if k_cap > 0:
            col_capacity = n_out * k_cap
        elif not sync:
            raise ValueError("an uncapped search without synchronisation needs col_capacity")
        else:
            col_capacity = max(1, 16 * n_out)
    lib = L.lib()
    ws = _Workspace(lib.sbc_points_workspace_size(n_in, n_out, n_batch, int(k_cap)), dev)
    row_ptr = torch.empty(n_out + 1, dtype=torch.int32, device=dev)
    stream = _stream(dev)
    for _ in range(2):
        col_idx = torch.empty(max(1, col_capacity), dtype=torch.int32, device=dev)
        nnz = ctypes.c_int64(-1)
        st = lib.sbc_neighbour_search_points(
            _p(x_in), n_in, _p(in_splits), _p(x_out), n_out, _p(out_splits), n_batch,
            ctypes.c_float(radius), int(k_cap), _p(row_ptr), _p(col_idx), int(col_capacity),
            ctypes.byref(nnz) if sync else None, ws.ptr, ws.nbytes, stream)
        if st == 2 and sync:          # capacity: retry once with the exact size
            col_capacity = int(nnz.value)
            continue
        L.check(st)
        E = int(nnz.value) if sync else int(col_capacity)
        return CSR(row_ptr, col_idx, n_out, n_in, E)
    raise RuntimeError("neighbour search did not converge on a capacity")


def _search_events(px, py, t, width, height, window, half_extent, col_capacity, sync, csc):
    _require(px, "px", torch.int32, 1)
    dev = px.device
    _require(py, "py", torch.int32, 1, dev)
    _require(t, "t", torch.int32, 1, dev)
    n = px.numel()
    if py.numel() != n or t.numel() != n:
        raise ValueError("px, py, t must have the same length")
    if col_capacity is None:
        if not sync:
            raise ValueError("sync=False needs col_capacity")
        col_capacity = max(1, 16 * n)
    lib = L.lib()
    ws = _Workspace(lib.sbc_events_workspace_size(n, width, height), dev)
    row_ptr = torch.empty(n + 1, dtype=torch.int32, device=dev)
    col_ptr = torch.empty(n + 1, dtype=torch.int32, device=dev) if csc else None
    stream = _stream(dev)
    for _ in range(2):
        col_idx = torch.empty(max(1, col_capacity), dtype=torch.int32, device=dev)
        nnz = ctypes.c_int64(-1)
        nnz_p = ctypes.byref(nnz) if sync else None
        common = (_p(px), _p(py), _p(t), n, int(width), int(height), int(half_extent), int(window),
                  _p(row_ptr), _p(col_idx))
        if csc:
            row_idx = torch.empty(max(1, col_capacity), dtype=torch.int32, device=dev)
            st = lib.sbc_neighbour_search_events_csc(*common, _p(col_ptr), _p(row_idx),
                                                     int(col_capacity), nnz_p, ws.ptr, ws.nbytes,
                                                     stream)
        else:
            st = lib.sbc_neighbour_search_events(*common, int(col_capacity), nnz_p, ws.ptr,
                                                 ws.nbytes, stream)
        if st == 2 and sync:
            col_capacity = int(nnz.value)
            continue
        L.check(st)
        E = int(nnz.value) if sync else int(col_capacity)
        csr = CSR(row_ptr, col_idx, n, n, E)
        return (csr, CSC(col_ptr, row_idx, None, n)) if csc else csr
    raise RuntimeError("neighbour search did not converge on a capacity")


def neighbour_search_events(px, py, t, width: int, height: int, window: int,
                            half_extent: int = 1, col_capacity: Optional[int] = None,
                            sync: bool = True) -> CSR:
    """Backwards-in-time pixel-block neighbourhoods of an event stream (sbc_neighbour_search_events)."""
    return _search_events(px, py, t, width, height, window, half_extent, col_capacity, sync,
                          False)


def neighbour_search_events_csc(px, py, t, width: int, height: int, window: int,
                                half_extent: int = 1, col_capacity: Optional[int] = None,
                                sync: bool = True) -> Tuple[CSR, CSC]:
    """The event neighbourhoods and their transpose from one search
    (sbc_neighbour_search_events_csc); the CSC has no edge_perm."""
    return _search_events(px, py, t, width, height, window, half_extent, col_capacity, sync,
                          True)


def basis_eval(csr: CSR, geometry: Geometry) -> torch.Tensor:
    """Per-edge basis values v [E, M] float32 (sbc_basis_eval)."""
    dev = csr.row_ptr.device
    geometry.check(csr)
    v = torch.empty((max(csr.nnz, 0), geometry.M), dtype=torch.float32, device=dev)
    c, g = csr.c_struct(), geometry.c_struct()
    L.check(L.lib().sbc_basis_eval(ctypes.byref(c), ctypes.byref(g), _p(v), _stream(dev)))
    return v


def csr_transpose(csr: CSR) -> CSC:
    """Stable transpose of the pattern (sbc_csr_transpose)."""
    dev = csr.row_ptr.device
    lib = L.lib()
    ws = _Workspace(lib.sbc_transpose_workspace_size(csr.n_cols, csr.nnz), dev)
    col_ptr = torch.empty(csr.n_cols + 1, dtype=torch.int32, device=dev)
    row_idx = torch.empty(max(1, csr.nnz), dtype=torch.int32, device=dev)
    perm = torch.empty(max(1, csr.nnz), dtype=torch.int32, device=dev)
    c = csr.c_struct()
    L.check(lib.sbc_csr_transpose(ctypes.byref(c), _p(col_ptr), _p(row_idx), _p(perm), ws.ptr,
                                  ws.nbytes, _stream(dev)))
    return CSC(col_ptr, row_idx, perm, csr.n_cols)


def csr_transpose_batched(csr: CSR, row_splits, col_splits) -> CSC:
    """Transpose of a block-diagonal pattern, block by block (sbc_csr_transpose_batched).

    row_splits / col_splits: int32 device tensors [n_batch + 1] (for a point
    search, out_splits and in_splits)."""
    dev = csr.row_ptr.device
    _require(row_splits, "row_splits", torch.int32, 1, dev)
    _require(col_splits, "col_splits", torch.int32, 1, dev)
    n_batch = int(row_splits.numel()) - 1
    if n_batch < 1 or int(col_splits.numel()) != n_batch + 1:
        raise ValueError("row_splits and col_splits must have the same length (>= 2)")
    col_ptr = torch.empty(csr.n_cols + 1, dtype=torch.int32, device=dev)
    row_idx = torch.empty(max(1, csr.nnz), dtype=torch.int32, device=dev)
    perm = torch.empty(max(1, csr.nnz), dtype=torch.int32, device=dev)
    c = csr.c_struct()
    L.check(L.lib().sbc_csr_transpose_batched(ctypes.byref(c), _p(row_splits), _p(col_splits),
                                              n_batch, _p(col_ptr), _p(row_idx), _p(perm),
                                              _stream(dev)))
    return CSC(col_ptr, row_idx, perm, csr.n_cols)


def _dtype_code(F: torch.Tensor) -> int:
    if F.dtype == torch.float32:
        return L.SBC_F32
    if F.dtype == torch.bfloat16:
        return L.SBC_BF16
    raise ValueError(f"features must be float32 or bfloat16, got {F.dtype}")


def _conv_common(csr, F, W, v, geometry):
    dev = csr.row_ptr.device
    _require(F, "F", (torch.float32, torch.bfloat16), 2, dev)
    _require(W, "W", F.dtype, 3, dev)
    M, C_in, C_out = W.shape
    if F.shape != (csr.n_cols, C_in):
        raise ValueError(f"F must be [{csr.n_cols}, {C_in}], got {tuple(F.shape)}")
    if v is not None:
        _require(v, "v", torch.float32, 2, dev)
        if v.shape[1] != M:
            raise ValueError("v must be [E, M]")
    elif geometry is None:
        raise ValueError("either v or geometry is needed")
    if geometry is not None:
        geometry.check(csr)
    return dev, M, C_in, C_out


def conv_workspace_size(csr: CSR, M, C_in, C_out, dtype_code, order) -> int:
    return L.lib().sbc_conv_workspace_size(csr.n_rows, csr.n_cols, csr.nnz, M, C_in, C_out,
                                           dtype_code, ORDERS[order])


def conv_forward(csr: CSR, F, W, geometry: Optional[Geometry] = None, v=None,
                 order: str = "auto") -> torch.Tensor:
    """Y = sum_m N^(m) F W^(m), float32 [n_out, C_out] (sbc_conv_forward)."""
    dev, M, C_in, C_out = _conv_common(csr, F, W, v, geometry)
    dt = _dtype_code(F)
    Y = torch.empty((csr.n_rows, C_out), dtype=torch.float32, device=dev)
    ws = _Workspace(conv_workspace_size(csr, M, C_in, C_out, dt, order), dev)
    c = csr.c_struct()
    g = geometry.c_struct() if geometry is not None else None
    L.check(L.lib().sbc_conv_forward(
        ctypes.byref(c), _p(v), ctypes.byref(g) if g is not None else None, M, _p(F), _p(W), dt,
        C_in, C_out, _p(Y), ORDERS[order], ws.ptr, ws.nbytes, _stream(dev)))
    return Y


def conv_forward_noalloc(csr: CSR, F, W, Y, geometry: Optional[Geometry] = None, v=None,
                         order: str = "auto") -> torch.Tensor:
    """The forward into a caller-given Y [n_out, C_out] float32, with the
    library's static scratch as its temporary space (sbc_conv_forward_noalloc):
    nothing is allocated, by this binding or by the library."""
    dev, M, C_in, C_out = _conv_common(csr, F, W, v, geometry)
    _require(Y, "Y", torch.float32, 2, dev)
    if tuple(Y.shape) != (csr.n_rows, C_out):
        raise ValueError(f"Y must be [{csr.n_rows}, {C_out}], got {tuple(Y.shape)}")
    c = csr.c_struct()
    g = geometry.c_struct() if geometry is not None else None
    L.check(L.lib().sbc_conv_forward_noalloc(
        ctypes.byref(c), _p(v), ctypes.byref(g) if g is not None else None, M, _p(F), _p(W),
        _dtype_code(F), C_in, C_out, _p(Y), ORDERS[order], _stream(dev)))
    return Y


def conv_forward_noalloc_max_bytes() -> int:
    """Bytes of the static scratch sbc_conv_forward_noalloc works in."""
    return int(L.lib().sbc_conv_forward_noalloc_max_bytes())


def conv_backward(csr: CSR, csc: CSC, F, W, dY, geometry: Optional[Geometry] = None, v=None,
                  order: str = "auto", need_dF: bool = True, need_dW: bool = True):
    """(dF [n_in, C_in], dW [M, C_in, C_out]) float32 (sbc_conv_backward)."""
    dev, M, C_in, C_out = _conv_common(csr, F, W, v, geometry)
    _require(dY, "dY", F.dtype, 2, dev)
    if dY.shape != (csr.n_rows, C_out):
        raise ValueError(f"dY must be [{csr.n_rows}, {C_out}]")
    dt = _dtype_code(F)
    dF = torch.empty((csr.n_cols, C_in), dtype=torch.float32, device=dev) if need_dF else None
    dW = torch.empty((M, C_in, C_out), dtype=torch.float32, device=dev) if need_dW else None
    ws = _Workspace(conv_workspace_size(csr, M, C_in, C_out, dt, order), dev)
    c, k = csr.c_struct(), csc.c_struct()
    g = geometry.c_struct() if geometry is not None else None
    L.check(L.lib().sbc_conv_backward(
        ctypes.byref(c), ctypes.byref(k), _p(v), ctypes.byref(g) if g is not None else None, M,
        _p(F), _p(W), _p(dY), dt, C_in, C_out, _p(dF), _p(dW), ORDERS[order], ws.ptr, ws.nbytes,
        _stream(dev)))
    return dF, dW


def _featureless_common(csr: CSR, M: int, geometry: Optional[Geometry], v):
    dev = csr.row_ptr.device
    if v is not None:
        _require(v, "v", torch.float32, 2, dev)
        if v.shape[1] != M:
            raise ValueError("v must be [E, M]")
    elif geometry is None:
        raise ValueError("either v or geometry is needed")
    if geometry is not None:
        geometry.check(csr)
    g = geometry.c_struct() if geometry is not None else None
    return dev, g


def featureless_forward(csr: CSR, Phi, geometry: Optional[Geometry] = None,
                        v=None) -> torch.Tensor:
    """Z = G~ Phi, float32 [n_out, P] (sbc_featureless_forward); Phi [M, P] float32."""
    _require(Phi, "Phi", torch.float32, 2, csr.row_ptr.device)
    M, P = Phi.shape
    dev, g = _featureless_common(csr, M, geometry, v)
    Z = torch.empty((csr.n_rows, P), dtype=torch.float32, device=dev)
    c = csr.c_struct()
    L.check(L.lib().sbc_featureless_forward(
        ctypes.byref(c), _p(v), ctypes.byref(g) if g is not None else None, M, _p(Phi), P,
        _p(Z), _stream(dev)))
    return Z


def featureless_backward(csr: CSR, dZ, M: int, geometry: Optional[Geometry] = None,
                         v=None) -> torch.Tensor:
    """dPhi = G~^T dZ, float32 [M, P] (sbc_featureless_backward)."""
    _require(dZ, "dZ", torch.float32, 2, csr.row_ptr.device)
    if dZ.shape[0] != csr.n_rows:
        raise ValueError(f"dZ must have {csr.n_rows} rows")
    P = dZ.shape[1]
    dev, g = _featureless_common(csr, M, geometry, v)
    dPhi = torch.empty((M, P), dtype=torch.float32, device=dev)
    lib = L.lib()
    ws = _Workspace(lib.sbc_featureless_workspace_size(csr.n_rows, M, P), dev)
    c = csr.c_struct()
    L.check(lib.sbc_featureless_backward(
        ctypes.byref(c), _p(v), ctypes.byref(g) if g is not None else None, M, _p(dZ), P,
        _p(dPhi), ws.ptr, ws.nbytes, _stream(dev)))
    return dPhi


def conv_decay_gradient(csr: CSR, F, W, dY, geometry: Geometry,
                        csc: Optional[CSC] = None) -> torch.Tensor:
    """d<Y, dY>/d lambda [M] float32 for the learned-decay event kernel
    (sbc_conv_decay_gradient); with the transpose it takes the fused route."""
    dev, M, C_in, C_out = _conv_common(csr, F, W, None, geometry)
    _require(dY, "dY", F.dtype, 2, dev)
    dt = _dtype_code(F)
    dl = torch.empty(M, dtype=torch.float32, device=dev)
    lib = L.lib()
    ws = _Workspace(lib.sbc_decay_gradient_workspace_size(csr.n_rows, csr.nnz, M, C_in, C_out,
                                                          dt), dev)
    c, g = csr.c_struct(), geometry.c_struct()
    k = csc.c_struct() if csc is not None else None
    L.check(lib.sbc_conv_decay_gradient(ctypes.byref(c), ctypes.byref(k) if k is not None else None,
                                        ctypes.byref(g), M, _p(F), _p(W), _p(dY), dt, C_in, C_out,
                                        _p(dl), ws.ptr, ws.nbytes, _stream(dev)))
    return dl


SAMPLING = {"ifp": 0, "approx_ifp": 1, "rejection": 2, "approx_ifp_rejection": 3}


def sample_points(x, splits, method: str, per_cloud: int = 0, ball: Optional[CSR] = None,
                  max_cloud: Optional[int] = None, with_dmin: bool = False):
    """Subsample a ragged point batch (sbc_sample_points).

    Returns (out_idx, out_splits) or, with with_dmin, (out_idx, out_splits,
    dmin2); out_idx holds capacity for every point, cloud b's outputs are
    out_idx[out_splits[b]:out_splits[b+1]].  ball: the in-place uncapped ball
    CSR (not needed for "ifp"); max_cloud: the largest cloud (read from splits
    when None, which synchronises)."""
    _require(x, "x", torch.float32, 2)
    dev = x.device
    _require(splits, "splits", torch.int32, 1, dev)
    n = x.shape[0]
    n_batch = splits.numel() - 1
    if max_cloud is None:
        max_cloud = int(torch.diff(splits).max().item()) if n_batch > 0 else 0
    out_idx = torch.empty(max(1, n), dtype=torch.int32, device=dev)
    out_splits = torch.empty(n_batch + 1, dtype=torch.int32, device=dev)
    dmin2 = torch.empty(max(1, n), dtype=torch.float32, device=dev) if with_dmin else None
    lib = L.lib()
    ws = _Workspace(lib.sbc_sampling_workspace_size(n_batch), dev)
    c = ball.c_struct() if ball is not None else None
    L.check(lib.sbc_sample_points(_p(x), _p(splits), n_batch, n, int(max_cloud),
                                  ctypes.byref(c) if c is not None else None, SAMPLING[method],
                                  int(per_cloud), _p(out_idx), _p(out_splits), _p(dmin2), ws.ptr,
                                  ws.nbytes, _stream(dev)))
    return (out_idx, out_splits, dmin2) if with_dmin else (out_idx, out_splits)


def lif_sample_events(px, py, t, width: int, height: int, kernel: int = 3, stride: int = 2,
                      decay: float = 1000.0, v_thresh: float = 1.5, v_reset: float = -3.0,
                      capacity: Optional[int] = None, sync: bool = True):
    """The coarser event stream by leaky integrate-and-fire (sbc_lif_sample_events).

    Returns (x, y, t, src, count): output pixels on the ceil(width / stride) x
    ceil(height / stride) grid, times, the input event behind each, and the
    number of output events.  With sync (the default) the arrays are trimmed
    to that number and count is an int; without, they keep their capacity
    (default: the most events possible) and count is an int64 device tensor."""
    _require(px, "px", torch.int32, 1)
    dev = px.device
    _require(py, "py", torch.int32, 1, dev)
    _require(t, "t", torch.int32, 1, dev)
    n = int(px.numel())
    if int(py.numel()) != n or int(t.numel()) != n:
        raise ValueError("px, py and t must have the same length")
    lib = L.lib()
    nsd = (int(kernel) - 1) // max(int(stride), 1) + 1
    if capacity is None:
        capacity = n * nsd * nsd
    cap = max(1, int(capacity))
    out = [torch.empty(cap, dtype=torch.int32, device=dev) for _ in range(4)]
    count = torch.zeros(1, dtype=torch.int64, device=dev)
    ws = _Workspace(lib.sbc_lif_workspace_size(n, width, height, kernel, stride), dev)
    host = ctypes.c_int64(0)
    L.check(lib.sbc_lif_sample_events(_p(px), _p(py), _p(t), n, width, height, kernel, stride,
                                      float(decay), float(v_thresh), float(v_reset),
                                      _p(out[0]), _p(out[1]), _p(out[2]), _p(out[3]),
                                      int(capacity), _p(count),
                                      ctypes.byref(host) if sync else None, ws.ptr, ws.nbytes,
                                      _stream(dev)))
    if sync:
        k = int(host.value)
        return tuple(o[:k] for o in out) + (k,)
    return tuple(out) + (count,)


class EventStream:
    """The state of the event convolution's deployment form (Eq. 13-15) over
    a width x height sensor, zero at the start, and step(), which feeds one
    batch and returns its outputs Y [n, C_out].

    decays None: the fixed decay, rate 1/tau for every offset
    (sbc_event_stream_step); z [height * width, C_in], W [8, C_in, C_out].
    decays [8, M_v] float32 (learned rates lambda_uv, Eq. 12): one sum per
    basis function (sbc_event_stream_step_decays); z [height * width, 8 M_v,
    C_in], W [8 M_v, C_in, C_out], function m = u M_v + v.  z_time [height *
    width] int32 either way."""

    def __init__(self, width: int, height: int, C_in: int, tau: float = None, device="cuda",
                 decays: torch.Tensor = None):
        self.width, self.height, self.C_in, self.tau = int(width), int(height), int(C_in), tau
        npix = self.width * self.height
        if decays is None:
            if tau is None or not tau > 0:
                raise ValueError("tau > 0 expected without decays")
            self.decays, self.M = None, 8
            self.z = torch.zeros((npix, self.C_in), dtype=torch.float32, device=device)
        else:
            _require(decays, "decays", torch.float32, 2, torch.device(device))
            if decays.shape[0] != 8 or not 1 <= decays.shape[1] <= 4:
                raise ValueError("decays [8, M_v] with 1 <= M_v <= 4 expected")
            self.decays, self.M = decays.contiguous(), 8 * int(decays.shape[1])
            self.z = torch.zeros((npix, self.M, self.C_in), dtype=torch.float32, device=device)
        self.z_time = torch.zeros(npix, dtype=torch.int32, device=device)

    def step(self, px, py, t, F, W) -> torch.Tensor:
        dev = self.z.device
        _require(px, "px", torch.int32, 1, dev)
        _require(py, "py", torch.int32, 1, dev)
        _require(t, "t", torch.int32, 1, dev)
        _require(F, "F", torch.float32, 2, dev)
        _require(W, "W", torch.float32, 3, dev)
        n = int(px.numel())
        if int(py.numel()) != n or int(t.numel()) != n or F.shape != (n, self.C_in) \
                or W.shape[:2] != (self.M, self.C_in):
            raise ValueError(f"px, py, t [n], F [n, C_in] and W [{self.M}, C_in, C_out] expected")
        C_out = int(W.shape[2])
        Y = torch.empty((max(n, 1), C_out), dtype=torch.float32, device=dev)
        lib = L.lib()
        if self.decays is None:
            ws = _Workspace(lib.sbc_event_stream_workspace_size(n, self.width, self.height,
                                                                self.C_in, C_out), dev)
            L.check(lib.sbc_event_stream_step(_p(px), _p(py), _p(t), _p(F), n, self.width,
                                              self.height, float(self.tau), _p(W), self.C_in,
                                              C_out, _p(self.z), _p(self.z_time), _p(Y), ws.ptr,
                                              ws.nbytes, _stream(dev)))
        else:
            Mv = self.M // 8
            ws = _Workspace(lib.sbc_event_stream_decays_workspace_size(
                n, self.width, self.height, Mv, self.C_in, C_out), dev)
            L.check(lib.sbc_event_stream_step_decays(
                _p(px), _p(py), _p(t), _p(F), n, self.width, self.height, _p(self.decays), Mv,
                _p(W), self.C_in, C_out, _p(self.z), _p(self.z_time), _p(Y), ws.ptr, ws.nbytes,
                _stream(dev)))
        return Y[:n]


def conv_plan(n_out, n_in, nnz, M, C_in, C_out, dtype=torch.float32, order="auto") -> dict:
    """Route and fusion of forward and backward for a shape (sbc_conv_plan)."""
    plan = L.SbcConvPlan()
    code = L.SBC_BF16 if dtype == torch.bfloat16 else L.SBC_F32
    L.check(L.lib().sbc_conv_plan(n_out, n_in, nnz, M, C_in, C_out, code, ORDERS[order],
                                  ctypes.byref(plan)))
    names = {v: k for k, v in ORDERS.items()}
    return {"forward_order": names[plan.forward_order], "backward_order": names[plan.backward_order],
            "forward_fused": bool(plan.forward_fused), "backward_fused": bool(plan.backward_fused)}


def resolve_order(n_out, n_in, nnz, M, C_in, C_out, order="auto") -> str:
    code = L.lib().sbc_resolve_order(n_out, n_in, nnz, M, C_in, C_out, ORDERS[order])
    return {v: k for k, v in ORDERS.items()}[code]
