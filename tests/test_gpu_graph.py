"""The whole step (search, forward, transpose, backward) captured in a HIP graph.

The step never synchronises with the host and allocates no device memory
inside the library, so it can be captured.  Every replay must reproduce the
eager results bit for bit (the kernels are deterministic), also with other
eager work and synchronisations between replays.
"""
import numpy as np
import pytest
import torch

import workloads
from tests import gpu_common as G

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["points", "events", "points_batched", "events_csc",
                                  "weighted", "featureless"])
def test_graph_replays_match_eager(name):
    """Each variant is one of the step forms the benchmark times: the general
    transpose, the block-diagonal transpose, the transpose from the reverse
    event search, the weighted basis (materialised inside the forward), and
    the featureless convolution."""
    print(f"[graph] {name}", flush=True)
    if name.startswith("points"):
        w = workloads.small_points(seed=11, c_in=64, c_out=64)
    elif name == "weighted":
        w = workloads.small_points(seed=18, c_in=64, c_out=64, basis=workloads.BASIS_WMONO10)
    elif name == "featureless":
        w = workloads.small_points(seed=19, c_in=1, c_out=32, basis=workloads.BASIS_WMONO10)
    else:
        w = workloads.small_events(seed=12, c=32)
    t = G.to_device(w)
    geo = G.geometry(w, t)
    cap = G.search(w, t).nnz       # a capacity for the unsynchronised search
    Phi = t["W"][:, 0, :].contiguous()

    def step():
        csc = None
        if w["kind"] == "points":
            csr = G.sbc.neighbour_search_points(t["x_in"], t["in_splits"], t["x_out"],
                                                t["out_splits"], w["radius"], w["k_cap"],
                                                sync=False)
        elif name == "events_csc":
            csr, csc = G.sbc.neighbour_search_events_csc(t["px"], t["py"], t["t"], w["width"],
                                                         w["height"], w["window"],
                                                         col_capacity=cap, sync=False)
        else:
            csr = G.sbc.neighbour_search_events(t["px"], t["py"], t["t"], w["width"],
                                                w["height"], w["window"], col_capacity=cap,
                                                sync=False)
        if name == "featureless":
            Z = G.sbc.featureless_forward(csr, Phi, geometry=geo)
            dPhi = G.sbc.featureless_backward(csr, t["dY"], w["M"], geometry=geo)
            return csr.row_ptr, Z, dPhi
        Y = G.sbc.conv_forward(csr, t["F"], t["W"], geometry=geo)
        if csc is None:
            csc = (G.sbc.csr_transpose_batched(csr, t["out_splits"], t["in_splits"])
                   if name == "points_batched" else G.sbc.csr_transpose(csr))
        dF, dW = G.sbc.conv_backward(csr, csc, t["F"], t["W"], t["dY"], geometry=geo)
        return csr.row_ptr, Y, dF, dW

    eager = [x.cpu().numpy().copy() for x in step()]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        outs = step()
    for r in range(3):
        # unrelated eager work and a synchronisation between replays
        junk = torch.randn(1 << 16, device=G.DEV).sum()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(eager, outs):
            assert np.array_equal(a, b.cpu().numpy()), f"replay {r} differs"
        assert torch.isfinite(junk)


def test_lif_graph_replays_match_eager():
    """The unsynchronised LIF sampler (sort, cells, scan, emission) captured in
    a graph reproduces the eager output events and count on every replay."""
    print("[graph] lif", flush=True)
    px, py, t, _ = workloads.uniform_events(np.random.default_rng(47), 20_000, 34, 34, 30_000)
    args = [torch.from_numpy(a).to(G.DEV) for a in (px, py, t)]

    def step():
        return G.sbc.lif_sample_events(*args, 34, 34, 3, 2, 2000.0, 1.5, -3.0, sync=False)

    eager = [x.cpu().numpy().copy() for x in step()]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        outs = step()
    k = int(eager[4][0])
    assert k > 0
    for r in range(3):
        junk = torch.randn(1 << 16, device=G.DEV).sum()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert int(outs[4].item()) == k, f"replay {r}: count differs"
        for a, b in zip(eager[:4], outs[:4]):
            assert np.array_equal(a[:k], b.cpu().numpy()[:k]), f"replay {r} differs"
        assert torch.isfinite(junk)


@pytest.mark.parametrize("Mv", [0, 2])
def test_event_stream_graph_replays_match_eager(Mv):
    """Three batches of the deployment form (fixed decay, or two learned
    decays per offset), the state reset at the start, captured in a graph:
    every replay reproduces the eager outputs and final state bit for bit."""
    print(f"[graph] event stream Mv {Mv}", flush=True)
    rng = np.random.default_rng(51)
    n, Wd, H = 6000, 24, 18
    px, py, t, _ = workloads.uniform_events(rng, n, Wd, H, 40_000)
    M = 8 * max(Mv, 1)
    F = torch.from_numpy(rng.standard_normal((n, 8)).astype(np.float32)).to(G.DEV)
    W = torch.from_numpy((rng.standard_normal((M, 8, 16)) / 8).astype(np.float32)).to(G.DEV)
    ev = [torch.from_numpy(a).to(G.DEV) for a in (px, py, t)]
    if Mv:
        lam = torch.from_numpy(rng.uniform(1e-4, 1e-3, (8, Mv)).astype(np.float32)).to(G.DEV)
        st = G.sbc.EventStream(Wd, H, 8, device=G.DEV, decays=lam)
    else:
        st = G.sbc.EventStream(Wd, H, 8, 2500.0, device=G.DEV)

    def step():
        st.z.zero_()
        st.z_time.zero_()
        return [st.step(ev[0][a:b], ev[1][a:b], ev[2][a:b], F[a:b], W)
                for a, b in [(0, 1000), (1000, 4500), (4500, n)]] + [st.z, st.z_time]

    eager = [x.cpu().numpy().copy() for x in step()]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        outs = step()
    for r in range(3):
        junk = torch.randn(1 << 16, device=G.DEV).sum()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(eager, outs):
            assert np.array_equal(a, b.cpu().numpy()), f"replay {r} differs"
        assert torch.isfinite(junk)
