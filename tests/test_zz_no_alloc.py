"""The forward entry point that allocates nothing (its temporary space is the
library's static device scratch), through the C ABI, against the workspace
entry point on the same inputs and against the oracle: calls in a row whose
inputs shrink, on the fused event and point routes and on the separate-kernel
route, and the refusal of a forward whose temporary space exceeds the scratch.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from tests import gpu_common as G

pytestmark = pytest.mark.gpu

# (case, order): larger inputs first, each followed by a smaller one
SEQUENCE = [
    ("fz_ev32", "auto"),          # 5003 events, 32 channels: fused, packed events in the scratch
    ("fz_tiny_ev", "auto"),       # 150 events
    ("fz_ev_bf16", "auto"),       # 4099 events, 64 bf16 channels
    ("fz_tiny_bf16", "auto"),     # 70 events
    ("fz_pts64", "auto"),         # point batch, fused
    ("pts_mono4_odd", "auto"),    # odd channels: basis values and G in the scratch
    ("pts_down", "gemm_first"),   # H = F W in the scratch
    ("fz_tiny_pts", "gemm_first"),
]

SMALL = {
    "fz_ev32": lambda: workloads.small_events(seed=3, c=32, n=5003),
    "fz_tiny_ev": lambda: workloads.small_events(seed=5, c=32, n=150),
    "fz_ev_bf16": lambda: workloads.small_events(seed=4, c=64, dtype="bf16", n=4099),
    "fz_tiny_bf16": lambda: workloads.small_events(seed=6, c=64, dtype="bf16", n=70),
    "fz_pts64": lambda: workloads.small_points(seed=7, c_in=64, c_out=64),
    "pts_mono4_odd": lambda: workloads.small_points(seed=4, basis=workloads.BASIS_MONO4, c_in=5,
                                                    c_out=7, n_out=45),
    "pts_down": lambda: workloads.small_points(seed=1, n_out=60),
    "fz_tiny_pts": lambda: workloads.small_points(seed=12, n_clouds=1, n=90, c_in=64, c_out=64),
}


def _oracle_y(w):
    if w["kind"] == "points":
        rp, ci = oracle.points_csr(w["x_in"], w["in_splits"], w["x_out"], w["out_splits"],
                                   w["radius"], w["k_cap"])
        v = oracle.basis.point_values(w["basis"], w["x_in"], w["x_out"], rp, ci, w["radius"],
                                      w["M"])
    else:
        rp, ci = oracle.events_csr(w["px"], w["py"], w["t"], w["window"], 1, w["width"],
                                   w["height"])
        v = oracle.basis.event_values(w["basis"], w["px"], w["py"], w["t"], rp, ci, w["tau"],
                                      w.get("decays"))
    return oracle.conv.forward(rp, ci, v, w["F"], w["W"])


def test_noalloc_forward_matches_the_workspace_forward():
    for name, order in SEQUENCE:
        print(f"[noalloc] {name} {order}", flush=True)
        w = SMALL[name]()
        t = G.to_device(w)
        csr = G.search(w, t)
        geo = G.geometry(w, t)
        ref = G.sbc.conv_forward(csr, t["F"], t["W"], geometry=geo, order=order)
        Y = torch.full((csr.n_rows, t["W"].shape[2]), float("nan"), dtype=torch.float32,
                       device=G.DEV)
        G.sbc.conv_forward_noalloc(csr, t["F"], t["W"], Y, geometry=geo, order=order)
        torch.cuda.synchronize()
        got = Y.cpu().numpy()
        assert np.array_equal(got, ref.cpu().numpy()), name
        tol = G.TOL_BF16 if w["dtype"] == "bf16" else G.TOL_F32
        assert G.row_error(got, _oracle_y(w)) < tol, name


def test_noalloc_forward_refuses_more_than_its_scratch():
    """H = F W of a GEMM-first forward over 300k inputs (77 MB) exceeds the
    64 MiB scratch: refused with SBC_ERR_WORKSPACE, Y untouched."""
    n, M, C = 300_000, 8, 32
    assert G.sbc.conv_forward_noalloc_max_bytes() == 64 << 20
    rp = torch.zeros(n + 1, dtype=torch.int32, device=G.DEV)
    ci = torch.zeros(1, dtype=torch.int32, device=G.DEV)
    csr = G.sbc.CSR(rp, ci, n, n, 1)
    F = torch.ones((n, C), dtype=torch.float32, device=G.DEV)
    W = torch.ones((M, C, C), dtype=torch.float32, device=G.DEV)
    v = torch.zeros((1, M), dtype=torch.float32, device=G.DEV)  # (a 0-row tensor has no address)
    Y = torch.full((n, C), 7.0, dtype=torch.float32, device=G.DEV)
    with pytest.raises(G.sbc.ops.L.SbcError, match="WORKSPACE"):
        G.sbc.conv_forward_noalloc(csr, F, W, Y, v=v, order="gemm_first")
    torch.cuda.synchronize()
    assert bool(torch.all(Y == 7.0))
