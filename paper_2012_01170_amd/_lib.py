"""ctypes declarations of the sbconv C ABI (include/sbconv.h).

Loading never builds: a missing library raises, so nothing can silently fall
back to another implementation.
"""
from __future__ import annotations

import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsbconv.so")

# enums
SBC_OK = 0
STATUS_NAMES = {0: "SBC_OK", 1: "SBC_ERR_INVALID_ARG", 2: "SBC_ERR_CAPACITY",
                3: "SBC_ERR_OVERFLOW", 4: "SBC_ERR_UNSORTED", 5: "SBC_ERR_OUT_OF_RANGE",
                6: "SBC_ERR_WORKSPACE", 7: "SBC_ERR_HIP", 8: "SBC_ERR_UNSUPPORTED",
                9: "SBC_ERR_INTERNAL"}
SBC_F32, SBC_BF16 = 0, 1
SBC_BASIS_MONO4, SBC_BASIS_MONO8, SBC_BASIS_EVENT8, SBC_BASIS_WMONO10 = 0, 1, 2, 3
SBC_BASIS_EVENT_DECAYS = 4
SBC_ORDER_AUTO, SBC_ORDER_SPMM_FIRST, SBC_ORDER_GEMM_FIRST = 0, 1, 2

EXPORTS = [
    "sbc_last_error", "sbc_status_string", "sbc_basis_size",
    "sbc_points_workspace_size", "sbc_neighbour_search_points",
    "sbc_events_workspace_size", "sbc_neighbour_search_events",
    "sbc_neighbour_search_events_csc", "sbc_basis_eval",
    "sbc_transpose_workspace_size", "sbc_csr_transpose", "sbc_csr_transpose_batched",
    "sbc_conv_workspace_size", "sbc_conv_forward", "sbc_conv_backward",
    "sbc_resolve_order", "sbc_trace_kernel", "sbc_trace_clear", "sbc_kernel_names",
    "sbc_conv_plan", "sbc_featureless_workspace_size", "sbc_featureless_forward",
    "sbc_featureless_backward", "sbc_decay_gradient_workspace_size", "sbc_conv_decay_gradient",
    "sbc_sampling_workspace_size", "sbc_sample_points",
    "sbc_lif_workspace_size", "sbc_lif_sample_events",
    "sbc_event_stream_workspace_size", "sbc_event_stream_step",
    "sbc_event_stream_decays_workspace_size", "sbc_event_stream_step_decays",
    "sbc_conv_forward_noalloc_max_bytes", "sbc_conv_forward_noalloc",
]


class SbcCsr(ctypes.Structure):
    _fields_ = [("n_rows", ctypes.c_int32), ("n_cols", ctypes.c_int32),
                ("nnz_bound", ctypes.c_int64), ("row_ptr", ctypes.c_void_p),
                ("col_idx", ctypes.c_void_p)]


class SbcCsc(ctypes.Structure):
    _fields_ = [("n_cols", ctypes.c_int32), ("col_ptr", ctypes.c_void_p),
                ("row_idx", ctypes.c_void_p), ("edge_perm", ctypes.c_void_p)]


class SbcGeometry(ctypes.Structure):
    _fields_ = [("basis", ctypes.c_int), ("radius", ctypes.c_float), ("tau", ctypes.c_float),
                ("x_in", ctypes.c_void_p), ("x_out", ctypes.c_void_p), ("px", ctypes.c_void_p),
                ("py", ctypes.c_void_p), ("t", ctypes.c_void_p), ("decays", ctypes.c_void_p),
                ("n_decays", ctypes.c_int32)]


class SbcConvPlan(ctypes.Structure):
    _fields_ = [("forward_order", ctypes.c_int), ("backward_order", ctypes.c_int),
                ("forward_fused", ctypes.c_int32), ("backward_fused", ctypes.c_int32)]


class SbcError(RuntimeError):
    def __init__(self, status: int, message: str):
        self.status = status
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")


_lib = None

_vp, _i32, _i64, _f32, _sz = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float,
                              ctypes.c_size_t)
_csr_p = ctypes.POINTER(SbcCsr)
_csc_p = ctypes.POINTER(SbcCsc)
_geo_p = ctypes.POINTER(SbcGeometry)
_i64_p = ctypes.POINTER(ctypes.c_int64)

_SIGS = {
    "sbc_last_error": (ctypes.c_char_p, []),
    "sbc_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "sbc_basis_size": (_i32, [ctypes.c_int]),
    "sbc_points_workspace_size": (_sz, [_i32, _i32, _i32, _i32]),
    "sbc_neighbour_search_points": (ctypes.c_int, [_vp, _i32, _vp, _vp, _i32, _vp, _i32, _f32, _i32,
                                                   _vp, _vp, _i64, _i64_p, _vp, _sz, _vp]),
    "sbc_events_workspace_size": (_sz, [_i32, _i32, _i32]),
    "sbc_neighbour_search_events": (ctypes.c_int, [_vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp,
                                                   _vp, _i64, _i64_p, _vp, _sz, _vp]),
    "sbc_neighbour_search_events_csc": (ctypes.c_int, [_vp, _vp, _vp, _i32, _i32, _i32, _i32,
                                                       _i32, _vp, _vp, _vp, _vp, _i64, _i64_p,
                                                       _vp, _sz, _vp]),
    "sbc_basis_eval": (ctypes.c_int, [_csr_p, _geo_p, _vp, _vp]),
    "sbc_featureless_workspace_size": (_sz, [_i32, _i32, _i32]),
    "sbc_sampling_workspace_size": (_sz, [_i32]),
    "sbc_sample_points": (ctypes.c_int, [_vp, _vp, _i32, _i32, _i32, _csr_p, ctypes.c_int, _i32,
                                         _vp, _vp, _vp, _vp, _sz, _vp]),
    "sbc_lif_workspace_size": (_sz, [_i32, _i32, _i32, _i32, _i32]),
    "sbc_lif_sample_events": (ctypes.c_int, [_vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32,
                                             ctypes.c_double, ctypes.c_double, ctypes.c_double,
                                             _vp, _vp, _vp, _vp, _i64, _vp, _i64_p, _vp, _sz,
                                             _vp]),
    "sbc_event_stream_workspace_size": (_sz, [_i32, _i32, _i32, _i32, _i32]),
    "sbc_event_stream_step": (ctypes.c_int, [_vp, _vp, _vp, _vp, _i32, _i32, _i32, _f32, _vp,
                                             _i32, _i32, _vp, _vp, _vp, _vp, _sz, _vp]),
    "sbc_event_stream_decays_workspace_size": (_sz, [_i32, _i32, _i32, _i32, _i32, _i32]),
    "sbc_event_stream_step_decays": (ctypes.c_int, [_vp, _vp, _vp, _vp, _i32, _i32, _i32, _vp,
                                                    _i32, _vp, _i32, _i32, _vp, _vp, _vp, _vp,
                                                    _sz, _vp]),
    "sbc_decay_gradient_workspace_size": (_sz, [_i32, _i64, _i32, _i32, _i32, ctypes.c_int]),
    "sbc_conv_decay_gradient": (ctypes.c_int, [_csr_p, _csc_p, _geo_p, _i32, _vp, _vp, _vp,
                                               ctypes.c_int, _i32, _i32, _vp, _vp, _sz, _vp]),
    "sbc_featureless_forward": (ctypes.c_int, [_csr_p, _vp, _geo_p, _i32, _vp, _i32, _vp, _vp]),
    "sbc_featureless_backward": (ctypes.c_int, [_csr_p, _vp, _geo_p, _i32, _vp, _i32, _vp, _vp,
                                                _sz, _vp]),
    "sbc_transpose_workspace_size": (_sz, [_i32, _i64]),
    "sbc_csr_transpose": (ctypes.c_int, [_csr_p, _vp, _vp, _vp, _vp, _sz, _vp]),
    "sbc_csr_transpose_batched": (ctypes.c_int, [_csr_p, _vp, _vp, _i32, _vp, _vp, _vp, _vp]),
    "sbc_conv_workspace_size": (_sz, [_i32, _i32, _i64, _i32, _i32, _i32, ctypes.c_int,
                                      ctypes.c_int]),
    "sbc_conv_forward": (ctypes.c_int, [_csr_p, _vp, _geo_p, _i32, _vp, _vp, ctypes.c_int, _i32,
                                        _i32, _vp, ctypes.c_int, _vp, _sz, _vp]),
    "sbc_conv_forward_noalloc_max_bytes": (_sz, []),
    "sbc_conv_forward_noalloc": (ctypes.c_int, [_csr_p, _vp, _geo_p, _i32, _vp, _vp, ctypes.c_int,
                                                _i32, _i32, _vp, ctypes.c_int, _vp]),
    "sbc_conv_backward": (ctypes.c_int, [_csr_p, _csc_p, _vp, _geo_p, _i32, _vp, _vp, _vp,
                                         ctypes.c_int, _i32, _i32, _vp, _vp, ctypes.c_int, _vp,
                                         _sz, _vp]),
    "sbc_resolve_order": (ctypes.c_int, [_i32, _i32, _i64, _i32, _i32, _i32, ctypes.c_int]),
    "sbc_trace_kernel": (ctypes.c_int, [ctypes.c_char_p, _vp, _vp]),
    "sbc_trace_clear": (None, []),
    "sbc_kernel_names": (ctypes.c_char_p, []),
    "sbc_conv_plan": (ctypes.c_int, [_i32, _i32, _i64, _i32, _i32, _i32, ctypes.c_int, ctypes.c_int,
                                     ctypes.POINTER(SbcConvPlan)]),
}


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2012_01170_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def check(status: int) -> None:
    if status != SBC_OK:
        msg = lib().sbc_last_error().decode(errors="replace")
        raise SbcError(status, msg)
