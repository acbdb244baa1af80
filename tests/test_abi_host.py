"""The C ABI without a GPU: exports, size queries, argument errors, order rule.

Nothing here launches a kernel; every call returns before touching the device.
"""
import ctypes
import os
import re

import pytest

from paper_2012_01170_amd import _lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(L.LIB_PATH):
        from paper_2012_01170_amd import build
        build.build()
    return L.lib()


def _declared():
    with open(os.path.join(ROOT, "include", "sbconv.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(sbc_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(lib):
    names = _declared()
    assert len(names) >= 14
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(L.EXPORTS) == names


def test_workspace_queries(lib):
    a = lib.sbc_points_workspace_size(32768, 32768, 32, 0)
    b = lib.sbc_points_workspace_size(1024, 256, 1, 0)
    assert a > b > 0 and a % 256 == 0
    # a capped search keeps n_out rows of k_cap entries
    assert lib.sbc_points_workspace_size(32768, 32768, 32, 32) >= a + 32768 * 32 * 4
    assert lib.sbc_events_workspace_size(300000, 128, 128) > 300000 * 4 * 5
    assert lib.sbc_transpose_workspace_size(1000, 5000) >= 2 * 5000 * 4
    s1 = lib.sbc_conv_workspace_size(1000, 1000, 8000, 8, 16, 16, L.SBC_F32, L.SBC_ORDER_SPMM_FIRST)
    s2 = lib.sbc_conv_workspace_size(1000, 1000, 8000, 8, 16, 16, L.SBC_F32, L.SBC_ORDER_GEMM_FIRST)
    assert s1 > 8000 * 8 * 4 and s2 > 8000 * 8 * 4
    assert lib.sbc_conv_workspace_size(-1, 10, 10, 8, 1, 1, 0, 0) == 0
    # the learned-decay stream keeps M = 8 M_v gathered rows per event
    s8 = lib.sbc_event_stream_workspace_size(4096, 128, 128, 32, 32)
    s16 = lib.sbc_event_stream_decays_workspace_size(4096, 128, 128, 2, 32, 32)
    assert s8 > 4096 * 8 * 32 * 4 and s16 >= s8 + 4096 * 8 * 32 * 4
    assert lib.sbc_event_stream_decays_workspace_size(4096, 128, 128, 1, 32, 32) >= s8
    assert lib.sbc_event_stream_decays_workspace_size(4096, 128, 128, 5, 32, 32) == 0
    assert lib.sbc_event_stream_decays_workspace_size(4096, 128, 128, 0, 32, 32) == 0


def test_stream_decays_argument_errors(lib):
    """Refusals the library decides before any device work."""
    L.lib()
    st = lib.sbc_event_stream_step_decays(None, None, None, None, 0, 8, 8, None, 2, None, 4, 4,
                                          None, None, None, None, 0, None)
    assert st == 1 and b"decays" in lib.sbc_last_error()
    st = lib.sbc_event_stream_step_decays(None, None, None, None, 0, 8, 8, None, 5, None, 4, 4,
                                          None, None, None, None, 0, None)
    assert st == 1 and b"n_decays" in lib.sbc_last_error()


def test_basis_sizes_and_strings(lib):
    assert [lib.sbc_basis_size(b) for b in (0, 1, 2)] == [4, 8, 8]
    assert lib.sbc_basis_size(7) == 0
    assert lib.sbc_status_string(2) == b"insufficient col_idx capacity"


def _search_points(lib, **kw):
    args = dict(x_in=1, n_in=4, in_splits=1, x_out=1, n_out=2, out_splits=1, n_batch=1,
                radius=0.1, k_cap=0, row_ptr=1, col_idx=1, cap=8, nnz=None, ws=1, ws_bytes=1 << 30,
                stream=None)
    args.update(kw)
    return lib.sbc_neighbour_search_points(
        args["x_in"], args["n_in"], args["in_splits"], args["x_out"], args["n_out"],
        args["out_splits"], args["n_batch"], ctypes.c_float(args["radius"]), args["k_cap"],
        args["row_ptr"], args["col_idx"], args["cap"], args["nnz"], args["ws"], args["ws_bytes"],
        args["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(n_batch=0), 1), (dict(radius=0.0), 1), (dict(radius=float("nan")), 1),
    (dict(radius=-1.0), 1), (dict(n_in=-1), 1), (dict(row_ptr=None), 1),
    (dict(cap=-1), 1), (dict(col_idx=None), 1), (dict(ws_bytes=16), 6), (dict(ws=None), 6),
])
def test_point_search_argument_errors(lib, kw, status):
    assert _search_points(lib, **kw) == status
    assert lib.sbc_last_error() != b""


@pytest.mark.parametrize("kw,status", [
    (dict(width=0), 1), (dict(half_extent=4), 8), (dict(window=-1), 1), (dict(px=None), 1),
    (dict(ws_bytes=8), 6), (dict(width=1 << 16, height=1 << 16), 1),
])
def test_event_search_argument_errors(lib, kw, status):
    a = dict(px=1, py=1, t=1, n=10, width=8, height=8, half_extent=1, window=5, row_ptr=1,
             col_idx=1, cap=10, nnz=None, ws=1, ws_bytes=1 << 30, stream=None)
    a.update(kw)
    st = lib.sbc_neighbour_search_events(a["px"], a["py"], a["t"], a["n"], a["width"],
                                         a["height"], a["half_extent"], a["window"], a["row_ptr"],
                                         a["col_idx"], a["cap"], a["nnz"], a["ws"], a["ws_bytes"],
                                         a["stream"])
    assert st == status


def test_conv_argument_errors(lib):
    csr = L.SbcCsr(10, 10, 40, 1, 1)
    g = L.SbcGeometry(L.SBC_BASIS_MONO8, 0.1, 0.0, 1, 1, 0, 0, 0)
    # stand-in device addresses (never dereferenced: every call below fails
    # its argument checks first), 16-byte aligned like real arrays
    A = 1 << 20
    ok = dict(M=8, F=A, W=A, dt=0, ci=4, co=4, Y=A, order=0, ws=A, wsb=1 << 30)

    def fwd(**kw):
        a = dict(ok)
        a.update(kw)
        return lib.sbc_conv_forward(ctypes.byref(csr), None, ctypes.byref(g), a["M"], a["F"],
                                    a["W"], a["dt"], a["ci"], a["co"], a["Y"], a["order"], a["ws"],
                                    a["wsb"], None)

    assert fwd(M=6) == 8
    assert fwd(M=4) == 1            # basis has M = 8
    assert fwd(ci=0) == 1
    assert fwd(dt=5) == 1
    assert fwd(W=None) == 1
    assert fwd(Y=None) == 1
    assert fwd(wsb=8) == 6
    # rows move 16 bytes at a time: unaligned arrays are argument errors
    assert fwd(F=A + 4) == 1
    assert fwd(W=A + 8) == 1
    assert fwd(Y=A + 12) == 1
    bad = L.SbcCsr(10, 10, 1 << 31, 1, 1)
    assert lib.sbc_conv_forward(ctypes.byref(bad), None, ctypes.byref(g), 8, A, A, 0, 4, 4, A, 0,
                                A, 1 << 30, None) == 3
    ge = L.SbcGeometry(L.SBC_BASIS_EVENT8, 0.0, 0.0, 0, 0, 1, 1, 1)
    assert lib.sbc_conv_forward(ctypes.byref(csr), None, ctypes.byref(ge), 8, A, A, 0, 4, 4, A,
                                0, A, 1 << 30, None) == 1          # tau = 0
    csc = L.SbcCsc(9, 1, 1, 1)                                      # n_cols mismatch
    assert lib.sbc_conv_backward(ctypes.byref(csr), ctypes.byref(csc), None, ctypes.byref(g), 8,
                                 A, A, A, 0, 4, 4, A, A, 0, A, 1 << 30, None) == 1
    csc = L.SbcCsc(10, 1, 1, 1)
    for dY, dF, dW in ((A + 4, A, A), (A, A + 4, A), (A, A, A + 4)):
        assert lib.sbc_conv_backward(ctypes.byref(csr), ctypes.byref(csc), None, ctypes.byref(g),
                                     8, A, A, dY, 0, 4, 4, dF, dW, 0, A, 1 << 30, None) == 1


@pytest.mark.parametrize("shape", [
    (256, 1024, 2800, 4, 16, 32), (32768, 32768, 194456, 8, 64, 64),
    (8192, 32768, 159867, 8, 64, 128), (32768, 8192, 159867, 8, 128, 64),
    (1000, 1000, 10, 8, 64, 8), (1000, 1000, 10, 8, 8, 64)])
def test_order_rule_is_the_cost_table(lib, shape):
    """AUTO picks the order with fewer multiply-adds (the paper's cost table)."""
    n_out, n_in, E, M, ci, co = shape
    spmm_first = M * ci * (E + n_out * co)
    gemm_first = M * co * (E + n_in * ci)
    want = L.SBC_ORDER_SPMM_FIRST if spmm_first <= gemm_first else L.SBC_ORDER_GEMM_FIRST
    assert lib.sbc_resolve_order(n_out, n_in, E, M, ci, co, L.SBC_ORDER_AUTO) == want
    assert lib.sbc_resolve_order(n_out, n_in, E, M, ci, co, L.SBC_ORDER_GEMM_FIRST) == 2


def test_trace_registry_without_events(lib):
    names = lib.sbc_kernel_names().decode().split(",")
    assert "fwd_gemm" in names and "points_fill" in names
    assert lib.sbc_trace_kernel(b"fwd_gemm", None, None) == 0     # removing is always fine
    assert lib.sbc_trace_kernel(None, None, None) == 1
    lib.sbc_trace_clear()


def test_conv_plan(lib):
    from paper_2012_01170_amd import ops
    p = ops.conv_plan(32768, 32768, 194456, 8, 64, 64)
    assert p == {"forward_order": "spmm_first", "backward_order": "spmm_first",
                 "forward_fused": True, "backward_fused": True}
    # down-sampling: gather first forward; the backward's cost rule picks dG first
    p = ops.conv_plan(8192, 32768, 159867, 8, 64, 128)
    assert p["forward_order"] == "spmm_first" and p["backward_order"] == "gemm_first"
    assert p["forward_fused"] and not p["backward_fused"]
    # a tiny problem: the multiply-adds favour dG first, but by less than the
    # three launches the fused D-route saves
    p = ops.conv_plan(256, 1024, 2894, 4, 16, 32)
    assert p["backward_order"] == "spmm_first" and p["backward_fused"]
    assert lib.sbc_resolve_order(1024, 256, 2894, 4, 32, 16, L.SBC_ORDER_AUTO) == \
        L.SBC_ORDER_GEMM_FIRST
    p = ops.conv_plan(100, 100, 500, 8, 5, 7)
    assert not p["forward_fused"] and not p["backward_fused"]
    p = ops.conv_plan(100, 100, 500, 8, 64, 64, order="gemm_first")
    assert p["forward_order"] == "gemm_first" and not p["forward_fused"]
    assert p["backward_order"] == "gemm_first" and not p["backward_fused"]


def test_noalloc_forward_refusals(lib):
    """The forward without a workspace reports its scratch size, checks its
    arguments like the workspace forward, and refuses, before touching the
    device, a forward whose temporary space exceeds the scratch."""
    assert lib.sbc_conv_forward_noalloc_max_bytes() == 64 << 20
    A = 1 << 20                     # stand-in device addresses, never dereferenced
    g = L.SbcGeometry(L.SBC_BASIS_MONO8, 0.1, 0.0, 1, 1, 0, 0, 0)
    csr = L.SbcCsr(10, 10, 40, 1, 1)
    assert lib.sbc_conv_forward_noalloc(ctypes.byref(csr), None, ctypes.byref(g), 6, A, A, 0, 4,
                                        4, A, 0, None) == 8
    assert lib.sbc_conv_forward_noalloc(ctypes.byref(csr), None, ctypes.byref(g), 8, A + 4, A, 0,
                                        4, 4, A, 0, None) == 1
    # GEMM-first over 300k inputs: H alone is 300k x 8 x 32 floats (77 MB)
    big = L.SbcCsr(300_000, 300_000, 0, 1, 1)
    assert lib.sbc_conv_forward_noalloc(ctypes.byref(big), A, None, 8, A, A, 0, 32, 32, A,
                                        L.SBC_ORDER_GEMM_FIRST, None) == 6
    assert b"static scratch" in lib.sbc_last_error()
