"""HIP path vs the CPU oracle, element by element, through the C ABI.

Neighbour CSRs and transposes must be bit-exact; basis values, outputs and
gradients must match to the float32 tolerance (bf16 inputs: the bf16 one),
row-normwise (gpu_common.row_error); rows that are exactly zero in the oracle
must be exactly zero.  Small cases span several tiles and a ragged tail;
the full-size workloads are checked on every CSR entry and on every row of
the outputs and gradients.
"""
import functools

import numpy as np
import pytest
import torch

import oracle
import workloads
from tests import gpu_common as G

pytestmark = pytest.mark.gpu

SMALL = {
    "pts_inplace": lambda: workloads.small_points(seed=0),
    "pts_down": lambda: workloads.small_points(seed=1, n_out=60),
    "pts_uncapped": lambda: workloads.small_points(seed=2, k_cap=0),
    "pts_cap1": lambda: workloads.small_points(seed=3, k_cap=1),
    "pts_mono4_odd": lambda: workloads.small_points(seed=4, basis=workloads.BASIS_MONO4, c_in=5,
                                                    c_out=7, n_out=45),
    "pts_wide": lambda: workloads.small_points(seed=5, n_clouds=2, c_in=96, c_out=80),
    "pts_bf16": lambda: workloads.small_points(seed=6, dtype="bf16", c_in=32, c_out=48),
    "ev_small": lambda: workloads.small_events(seed=0),
    "ev_odd": lambda: workloads.small_events(seed=1, c=13, n=3001),
    "ev_bf16": lambda: workloads.small_events(seed=2, dtype="bf16", c=24),
    # shapes with fused kernels, at sizes spanning several tiles and a ragged tail
    "fz_pts64": lambda: workloads.small_points(seed=7, c_in=64, c_out=64),
    "fz_pts_down128": lambda: workloads.small_points(seed=8, n_out=61, c_in=64, c_out=128),
    "fz_pts_m4": lambda: workloads.small_points(seed=9, basis=workloads.BASIS_MONO4, n_out=70,
                                                c_in=16, c_out=32),
    "fz_pts_bf16": lambda: workloads.small_points(seed=10, dtype="bf16", c_in=32, c_out=32),
    "fz_ev32": lambda: workloads.small_events(seed=3, c=32, n=5003),
    "fz_ev_bf16": lambda: workloads.small_events(seed=4, c=64, dtype="bf16", n=4099),
    # fewer tiles than XCDs / persistent blocks
    "fz_tiny_ev": lambda: workloads.small_events(seed=5, c=32, n=150),
    "fz_tiny_pts": lambda: workloads.small_points(seed=12, n_clouds=1, n=90, c_in=64, c_out=64),
    "fz_tiny_bf16": lambda: workloads.small_events(seed=6, c=64, dtype="bf16", n=70),
    "fz_tiny_bf16_32": lambda: workloads.small_events(seed=13, c=32, dtype="bf16", n=70),
    # the weighted convolution with M = 10 (unfused routes)
    "pts_weighted": lambda: workloads.small_points(seed=14, basis=workloads.BASIS_WMONO10,
                                                   c_in=16, c_out=24),
    "pts_weighted_odd": lambda: workloads.small_points(seed=15, n_out=50, k_cap=0, c_in=5,
                                                       c_out=7, basis=workloads.BASIS_WMONO10),
    "pts_weighted_bf16": lambda: workloads.small_points(seed=16, basis=workloads.BASIS_WMONO10,
                                                        c_in=32, c_out=32, dtype="bf16"),
    "fz_pts_weighted64": lambda: workloads.small_points(seed=17, basis=workloads.BASIS_WMONO10,
                                                        c_in=64, c_out=64),
    # the event kernel with learned decays (M_v = 2, 3, 4 per offset; unfused routes)
    "ev_decays2": lambda: workloads.small_events(seed=20, c=8, n_decays=2),
    "ev_decays3_odd": lambda: workloads.small_events(seed=22, n=3001, c=13, n_decays=3),
    "ev_decays4_bf16": lambda: workloads.small_events(seed=21, c=16, n_decays=4, dtype="bf16"),
    "fz_ev_decays2_32": lambda: workloads.small_events(seed=23, c=32, n=5003, n_decays=2),
    # uncapped wide balls: rows and columns of more than 64 edges with a ragged
    # tail (the generic gathers fetch a row's edges 64 at a time)
    "pts_dense": lambda: workloads.small_points(seed=24, n_clouds=2, n=200, radius=0.9, k_cap=0,
                                                c_in=16, c_out=24),
}
# the general convolution's full-size cases; the featureless first layer
# (one input channel of features ~N(0,1), so single-channel input gradients
# whose sums cancel by up to 1e6) is checked as Eq. 9-10 instead
FULL = [k for k in workloads.WORKLOADS
        if k not in ("ellipsoids_featureless", "ellipsoids_sampling", "events_300k_lif",
                     "events_stream")]
ORDERS = ["spmm_first", "gemm_first"]


@functools.lru_cache(maxsize=None)
def case(name):
    w = SMALL[name]() if name in SMALL else workloads.WORKLOADS[name]()
    if w["kind"] == "points":
        rp, ci = oracle.points_csr(w["x_in"], w["in_splits"], w["x_out"], w["out_splits"],
                                   w["radius"], w["k_cap"])
        v = oracle.basis.point_values(w["basis"], w["x_in"], w["x_out"], rp, ci, w["radius"], w["M"])
    else:
        rp, ci = oracle.events_csr(w["px"], w["py"], w["t"], w["window"], 1, w["width"],
                                   w["height"])
        v = oracle.basis.event_values(w["basis"], w["px"], w["py"], w["t"], rp, ci,
                                      w["tau"], w.get("decays"))
    return w, rp, ci, v


@functools.lru_cache(maxsize=None)
def gpu_case(name):
    w, rp, ci, v = case(name)
    t = G.to_device(w)
    csr = G.search(w, t)
    return t, csr


@functools.lru_cache(maxsize=2)
def oracle_forward(name):
    """Every row of Y from the oracle (the full-size event streams take seconds)."""
    w, rp, ci, v = case(name)
    print(f"    oracle forward {name}", flush=True)
    return oracle.conv.forward(rp, ci, v, w["F"], w["W"])


@functools.lru_cache(maxsize=2)
def oracle_backward(name):
    """Every row of dF, and dW, from the oracle."""
    w, rp, ci, v = case(name)
    print(f"    oracle backward {name}", flush=True)
    return oracle.conv.backward(rp, ci, v, w["F"], w["W"], w["dY"], w["n_in"])


def tol(w):
    return G.TOL_BF16 if w["dtype"] == "bf16" else G.TOL_F32


# ---------------------------------------------------------------- neighbours
@pytest.mark.parametrize("name", list(SMALL) + FULL)
def test_csr_bit_exact(name):
    print(f"[csr] {name}", flush=True)
    w, rp, ci, _ = case(name)
    t, csr = gpu_case(name)
    assert csr.nnz == len(ci)
    assert np.array_equal(csr.row_ptr.cpu().numpy(), rp)
    assert np.array_equal(csr.col_idx[:csr.nnz].cpu().numpy(), ci)


@pytest.mark.parametrize("name", ["pts_inplace", "pts_down", "ellipsoids_inplace"])
def test_csr_without_sync(name):
    print(f"[csr nosync] {name}", flush=True)
    w, rp, ci, _ = case(name)
    t = G.to_device(w)
    csr = G.search(w, t, sync=False)
    torch.cuda.synchronize()
    got_rp = csr.row_ptr.cpu().numpy()
    assert np.array_equal(got_rp, rp)
    assert np.array_equal(csr.col_idx[:got_rp[-1]].cpu().numpy(), ci)


def test_csr_transpose_bit_exact():
    for name in ["pts_down", "pts_uncapped", "ev_small", "ellipsoids_down", "events_300k"]:
        print(f"[transpose] {name}", flush=True)
        w, rp, ci, _ = case(name)
        t, csr = gpu_case(name)
        csc = G.sbc.csr_transpose(csr)
        cp, ri, perm = oracle.csr_transpose(rp, ci, w["n_in"])
        assert np.array_equal(csc.col_ptr.cpu().numpy(), cp)
        assert np.array_equal(csc.row_idx[:len(ci)].cpu().numpy(), ri)
        assert np.array_equal(csc.edge_perm[:len(ci)].cpu().numpy(), perm)


# ---------------------------------------------------------------- basis
@pytest.mark.parametrize("name", list(SMALL) + FULL)
def test_basis_values(name):
    print(f"[basis] {name}", flush=True)
    w, rp, ci, v_ref = case(name)
    t, csr = gpu_case(name)
    v = G.sbc.basis_eval(csr, G.geometry(w, t)).cpu().numpy()
    assert v.shape == v_ref.shape
    # all basis values are bounded by 1 in magnitude: absolute float32 error
    assert np.max(np.abs(v - v_ref)) < 2e-6
    assert np.all(v[v_ref == 0] == 0) or w["kind"] == "points"


# ---------------------------------------------------------------- forward
@pytest.mark.parametrize("order", ORDERS)
@pytest.mark.parametrize("name", list(SMALL) + FULL)
def test_forward(name, order):
    print(f"[forward] {name} {order}", flush=True)
    w, rp, ci, v = case(name)
    t, csr = gpu_case(name)
    Y = G.sbc.conv_forward(csr, t["F"], t["W"], geometry=G.geometry(w, t), order=order)
    err = G.row_error(Y.cpu().numpy(), oracle_forward(name))
    print(f"    row error {err:.3e}", flush=True)
    assert err < tol(w)


@pytest.mark.parametrize("name", ["pts_down", "ev_odd", "sphere_1024", "fz_pts64", "fz_ev32",
                                  "pts_weighted"])
def test_forward_with_materialised_basis(name):
    w, rp, ci, v = case(name)
    t, csr = gpu_case(name)
    vv = G.sbc.basis_eval(csr, G.geometry(w, t))
    for order in ORDERS:
        Y = G.sbc.conv_forward(csr, t["F"], t["W"], v=vv, order=order)
        Y_ref = oracle.conv.forward(rp, ci, v, w["F"], w["W"])
        assert G.row_error(Y.cpu().numpy(), Y_ref) < tol(w)


# ---------------------------------------------------------------- backward
@pytest.mark.parametrize("order", ORDERS)
@pytest.mark.parametrize("name", list(SMALL) + FULL)
def test_backward(name, order):
    print(f"[backward] {name} {order}", flush=True)
    w, rp, ci, v = case(name)
    t, csr = gpu_case(name)
    csc = G.sbc.csr_transpose(csr)
    dF, dW = G.sbc.conv_backward(csr, csc, t["F"], t["W"], t["dY"], geometry=G.geometry(w, t),
                                 order=order)
    dF_ref, dW_ref = oracle_backward(name)
    e1 = G.row_error(dF.cpu().numpy(), dF_ref)
    e2 = G.norm_error(dW.cpu().numpy(), dW_ref)
    print(f"    dF row error {e1:.3e}  dW error {e2:.3e}", flush=True)
    assert e1 < tol(w) and e2 < tol(w)


@pytest.mark.parametrize("name", ["pts_mono4_odd", "fz_pts64", "fz_ev_bf16"])
def test_backward_with_materialised_basis_and_partial_outputs(name):
    w, rp, ci, v = case(name)
    t, csr = gpu_case(name)
    csc = G.sbc.csr_transpose(csr)
    vv = G.sbc.basis_eval(csr, G.geometry(w, t))
    dF_ref, dW_ref = oracle.conv.backward(rp, ci, v, w["F"], w["W"], w["dY"], w["n_in"])
    for order in ORDERS:
        dF, dW = G.sbc.conv_backward(csr, csc, t["F"], t["W"], t["dY"], v=vv, order=order)
        assert G.row_error(dF.cpu().numpy(), dF_ref) < tol(w)
        assert G.norm_error(dW.cpu().numpy(), dW_ref) < tol(w)
        dF1, none = G.sbc.conv_backward(csr, csc, t["F"], t["W"], t["dY"], v=vv, order=order,
                                        need_dW=False)
        none2, dW1 = G.sbc.conv_backward(csr, csc, t["F"], t["W"], t["dY"], v=vv, order=order,
                                         need_dF=False)
        assert none is None and none2 is None
        assert np.array_equal(dF1.cpu().numpy(), dF.cpu().numpy())
        assert np.array_equal(dW1.cpu().numpy(), dW.cpu().numpy())


def test_runs_are_bitwise_reproducible():
    for name in ["ev_small", "pts_down", "fz_pts64", "fz_ev_bf16"]:
        w, rp, ci, v = case(name)
        t, csr = gpu_case(name)
        csc = G.sbc.csr_transpose(csr)
        g = G.geometry(w, t)
        outs = []
        for _ in range(2):
            Y = G.sbc.conv_forward(csr, t["F"], t["W"], geometry=g)
            dF, dW = G.sbc.conv_backward(csr, csc, t["F"], t["W"], t["dY"], geometry=g)
            outs.append([x.cpu().numpy() for x in (Y, dF, dW)])
        for a, b in zip(*outs):
            assert np.array_equal(a, b)


# ---------------------------------------------------------------- edge cases
def test_isolated_and_empty_outputs_are_exact_zero():
    w = workloads.small_points(seed=8, n_out=30, n_clouds=2)
    # an output far from everything, and a last cloud with no inputs
    w["x_out"] = np.concatenate([w["x_out"], np.array([[9, 9, 9]], np.float32)])
    w["out_splits"] = w["out_splits"].copy()
    w["out_splits"][-1] += 1
    w["dY"] = np.concatenate([w["dY"], np.ones((1, w["C_out"]), np.float32)])
    w["n_out"] += 1
    t = G.to_device(w)
    csr = G.search(w, t)
    Y = G.sbc.conv_forward(csr, t["F"], t["W"], geometry=G.geometry(w, t)).cpu().numpy()
    assert np.all(Y[-1] == 0.0)
    rp, ci = oracle.points_csr(w["x_in"], w["in_splits"], w["x_out"], w["out_splits"],
                               w["radius"], w["k_cap"])
    assert np.array_equal(csr.row_ptr.cpu().numpy(), rp)


POINT_CASES = ["pts_inplace", "pts_down", "pts_uncapped", "pts_cap1", "pts_mono4_odd", "pts_wide",
               "fz_pts64", "fz_pts_down128", "fz_tiny_pts", "sphere_1024", "ellipsoids_inplace",
               "ellipsoids_down"]


def check_transpose(csc, rp, ci, n_cols):
    cp, ri, perm = oracle.csr_transpose(rp, ci, n_cols)
    assert np.array_equal(csc.col_ptr.cpu().numpy(), cp)
    assert np.array_equal(csc.row_idx[:len(ci)].cpu().numpy(), ri)
    assert np.array_equal(csc.edge_perm[:len(ci)].cpu().numpy(), perm)


@pytest.mark.parametrize("name", POINT_CASES)
def test_batched_transpose_bit_exact(name):
    """Block-by-block transpose of a ragged batch's CSR equals the oracle's."""
    print(f"[transpose batched] {name}", flush=True)
    w, rp, ci, _ = case(name)
    t, csr = gpu_case(name)
    csc = G.sbc.csr_transpose_batched(csr, t["out_splits"], t["in_splits"])
    check_transpose(csc, rp, ci, w["n_in"])


def test_batched_transpose_large_blocks():
    """Windows halved when a block's columns hold more entries than the LDS
    stage, and single columns longer than the stage (rows past the staged
    row bounds too)."""
    rng = np.random.default_rng(3)
    x = (rng.random((1500, 3)) * 0.1).astype(np.float32)
    w = workloads.points_workload(rng, [(x, x[:40])], workloads.BASIS_MONO8, 0.3, 0, 4, 4)
    rp, ci = oracle.points_csr(w["x_in"], w["in_splits"], w["x_out"], w["out_splits"], 0.3, 0)
    assert len(ci) == 40 * 1500
    t = G.to_device(w)
    csr = G.search(w, t)
    check_transpose(G.sbc.csr_transpose_batched(csr, t["out_splits"], t["in_splits"]), rp, ci,
                    1500)
    # two blocks of 4500 rows, each row holding all 3 columns of its block
    n = 9000
    rp = np.arange(0, 3 * n + 1, 3, dtype=np.int32)
    ci = np.concatenate([np.arange(3) + (3 if r >= n // 2 else 0) for r in range(n)]).astype(np.int32)
    csr = G.sbc.CSR(G.dev(rp), G.dev(ci), n, 6, len(ci))
    splits_r = G.dev(np.array([0, n // 2, n], np.int32))
    splits_c = G.dev(np.array([0, 3, 6], np.int32))
    check_transpose(G.sbc.csr_transpose_batched(csr, splits_r, splits_c), rp, ci, 6)


@pytest.mark.parametrize("n_batch,k_cap,radius", [(70, 12, 0.35), (130, 0, 0.2), (63, 5, 0.3)])
def test_many_clouds(n_batch, k_cap, radius):
    """Batches of 63 to 130 clouds (the splits are read by the wave 64 at a
    time), with empty clouds among them."""
    print(f"[many clouds] {n_batch} k_cap {k_cap}", flush=True)
    rng = np.random.default_rng(n_batch)
    x = workloads.ellipsoid_surface_points(rng, 2400, np.array([1.0, 0.7, 0.5]))
    cuts = np.sort(rng.integers(0, len(x) + 1, size=n_batch - 1))
    cuts[:3] = cuts[3]            # a few empty clouds in a row
    splits = np.concatenate([[0], cuts, [len(x)]]).astype(np.int32)
    w = workloads.points_workload(rng, [(x, x)], workloads.BASIS_MONO8, radius, k_cap, 4, 4)
    w["in_splits"] = splits
    w["out_splits"] = splits.copy()
    rp, ci = oracle.points_csr(w["x_in"], w["in_splits"], w["x_out"], w["out_splits"],
                               w["radius"], k_cap)
    t = G.to_device(w)
    csr = G.search(w, t)
    assert np.array_equal(csr.row_ptr.cpu().numpy(), rp)
    assert np.array_equal(csr.col_idx[:csr.nnz].cpu().numpy(), ci)
    check_transpose(G.sbc.csr_transpose_batched(csr, t["out_splits"], t["in_splits"]), rp, ci,
                    len(x))


@pytest.mark.parametrize("sizes", [[5000] + [0] * 8 + [10], [1100, 1200]])
def test_cloud_table_builds(sizes):
    """Batches whose average cloud is small take the per-cloud table build: a
    5000-point cloud among empty ones counts in global memory there; a batch
    of larger clouds takes the multi-kernel build."""
    print(f"[cloud tables] {sizes}", flush=True)
    rng = np.random.default_rng(len(sizes))
    clouds = [workloads.ellipsoid_surface_points(rng, n, np.array([1.0, 0.8, 0.6])) if n else
              np.zeros((0, 3)) for n in sizes]
    w = workloads.points_workload(rng, [(x, x) for x in clouds], workloads.BASIS_MONO8, 0.08, 16,
                                  4, 4)
    rp, ci = oracle.points_csr(w["x_in"], w["in_splits"], w["x_out"], w["out_splits"], 0.08, 16)
    t = G.to_device(w)
    csr = G.search(w, t)
    assert np.array_equal(csr.row_ptr.cpu().numpy(), rp)
    assert np.array_equal(csr.col_idx[:csr.nnz].cpu().numpy(), ci)


def test_empty_stream_and_cloud():
    z = torch.zeros(0, dtype=torch.int32, device=G.DEV)
    csr = G.sbc.neighbour_search_events(z, z, z, 8, 8, 100)
    assert csr.nnz == 0 and csr.row_ptr.cpu().tolist() == [0]
    x = torch.zeros((0, 3), dtype=torch.float32, device=G.DEV)
    s = torch.zeros(2, dtype=torch.int32, device=G.DEV)
    csr = G.sbc.neighbour_search_points(x, s, x, s, 0.1, 4)
    assert csr.nnz == 0 and csr.row_ptr.cpu().tolist() == [0]


@pytest.mark.parametrize("k_cap", [0, 7, 300, 700])
def test_rows_longer_than_the_lds_stage(k_cap):
    """A dense cloud whose in-ball rows exceed the kernel's LDS stage (512)."""
    rng = np.random.default_rng(3)
    x = (rng.random((1500, 3)) * 0.1).astype(np.float32)
    y = x[:40]
    w = workloads.points_workload(rng, [(x, y)], workloads.BASIS_MONO8, 0.3, k_cap, 4, 4)
    rp, ci = oracle.points_csr(w["x_in"], w["in_splits"], w["x_out"], w["out_splits"],
                               w["radius"], k_cap)
    assert np.diff(rp).max() == (k_cap if k_cap else 1500)
    t = G.to_device(w)
    csr = G.search(w, t)
    assert np.array_equal(csr.row_ptr.cpu().numpy(), rp)
    assert np.array_equal(csr.col_idx[:csr.nnz].cpu().numpy(), ci)


@pytest.mark.parametrize("k_cap", [0, 16, 200, 300])
def test_two_rows_per_wave(k_cap):
    """Enough output rows (over 16384) that each wave searches two rows: a
    sparse cloud with a dense cluster (1500 points in ball) and a medium one
    (about 150), so that capped and uncapped rows take the staged, the
    bisection and the unstaged paths on 32-lane row segments."""
    print(f"[two rows per wave] k_cap {k_cap}", flush=True)
    rng = np.random.default_rng(11)
    dense = (rng.random((1500, 3)) * 0.1).astype(np.float32)
    medium = (rng.random((150, 3)) * 0.1 + 1.0).astype(np.float32)
    sparse = (rng.random((18500, 3)) * 10.0 + 2.0).astype(np.float32)
    x = np.concatenate([dense, medium, sparse])
    y = np.concatenate([dense[:40], medium[:40], sparse])
    w = workloads.points_workload(rng, [(x, y)], workloads.BASIS_MONO8, 0.3, k_cap, 4, 4)
    rp, ci = oracle.points_csr(w["x_in"], w["in_splits"], w["x_out"], w["out_splits"], 0.3, k_cap)
    lens = np.diff(rp)
    assert lens[0] == (k_cap if k_cap else 1500) and len(lens) > 16384
    t = G.to_device(w)
    csr = G.search(w, t)
    assert np.array_equal(csr.row_ptr.cpu().numpy(), rp)
    assert np.array_equal(csr.col_idx[:csr.nnz].cpu().numpy(), ci)


def test_weighted_basis_needs_edge_perm():
    """The weighted basis is normalised per output row, so a transpose without
    edge positions is refused (before anything is enqueued)."""
    w, rp, ci, v = case("pts_weighted")
    t, csr = gpu_case("pts_weighted")
    csc = G.sbc.csr_transpose(csr)
    bare = G.sbc.CSC(csc.col_ptr, csc.row_idx, None, csc.n_cols)
    with pytest.raises(G.sbc.ops.L.SbcError, match="INVALID_ARG"):
        G.sbc.conv_backward(csr, bare, t["F"], t["W"], t["dY"], geometry=G.geometry(w, t))


def test_weighted_rows_sum_to_one_on_the_gpu():
    """Partition of unity of the GPU's weighted values (Eq. 11): the constant
    basis function's values of every non-empty row sum to 1."""
    w, rp, ci, v = case("ellipsoids_weighted")
    t, csr = gpu_case("ellipsoids_weighted")
    vv = G.sbc.basis_eval(csr, G.geometry(w, t)).cpu().numpy().astype(np.float64)
    lens = np.diff(rp)
    sums = np.add.reduceat(vv[:, 0], rp[:-1][lens > 0])
    assert np.allclose(sums, 1.0, rtol=0, atol=1e-5)


def test_unsorted_and_out_of_range_events_are_reported():
    px = torch.tensor([1, 2, 3, 1], dtype=torch.int32, device=G.DEV)
    py = torch.tensor([1, 1, 1, 1], dtype=torch.int32, device=G.DEV)
    t = torch.tensor([0, 10, 5, 20], dtype=torch.int32, device=G.DEV)
    with pytest.raises(G.sbc.ops.L.SbcError, match="UNSORTED"):
        G.sbc.neighbour_search_events(px, py, t, 8, 8, 100)
    t2 = torch.tensor([0, 10, 15, 20], dtype=torch.int32, device=G.DEV)
    px2 = torch.tensor([1, 2, 8, 1], dtype=torch.int32, device=G.DEV)
    with pytest.raises(G.sbc.ops.L.SbcError, match="OUT_OF_RANGE"):
        G.sbc.neighbour_search_events(px2, py, t2, 8, 8, 100)


def test_malformed_splits_are_reported():
    x = torch.zeros((4, 3), dtype=torch.float32, device=G.DEV)
    good = torch.tensor([0, 4], dtype=torch.int32, device=G.DEV)
    bad = torch.tensor([0, 5], dtype=torch.int32, device=G.DEV)
    with pytest.raises(G.sbc.ops.L.SbcError, match="OUT_OF_RANGE"):
        G.sbc.neighbour_search_points(x, bad, x, good, 0.1, 2)


@pytest.mark.parametrize("n_cols", [5_000_000, 8192, 8193])
def test_transpose_of_wide_patterns(n_cols):
    """Column counts of 5M entries take the scan's recursive path; 8192/8193 its boundaries."""
    rng = np.random.default_rng(n_cols)
    n_rows = 3000
    lens = rng.integers(0, 9, size=n_rows)
    rp = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    ci = np.concatenate([np.sort(rng.choice(n_cols, size=k, replace=False)) for k in lens])
    ci = ci.astype(np.int32)
    csr = G.sbc.CSR(G.dev(rp), G.dev(ci), n_rows, n_cols, len(ci))
    csc = G.sbc.csr_transpose(csr)
    cp, ri, perm = oracle.csr_transpose(rp, ci, n_cols)
    assert np.array_equal(csc.col_ptr.cpu().numpy(), cp)
    assert np.array_equal(csc.row_idx[:len(ci)].cpu().numpy(), ri)
    assert np.array_equal(csc.edge_perm[:len(ci)].cpu().numpy(), perm)


@pytest.mark.parametrize("half_extent", [0, 1, 2, 3])
def test_event_search_block_sizes(half_extent):
    """1x1 and 3x3 blocks take the stored-run sweep, 5x5 and 7x7 the per-event bisection.

    A small sensor with a hot pixel gives long per-pixel lists and rows.
    """
    print(f"[events h={half_extent}]", flush=True)
    rng = np.random.default_rng(40 + half_extent)
    n, W, H = 6000, 9, 7
    px = rng.integers(0, W, size=n).astype(np.int32)
    py = rng.integers(0, H, size=n).astype(np.int32)
    hot = rng.random(n) < 0.2
    px[hot], py[hot] = 4, 3
    t = np.sort(rng.integers(0, 40_000, size=n)).astype(np.int32)
    window = 900
    rp, ci = oracle.events_csr(px, py, t, window, half_extent, W, H)
    csr = G.sbc.neighbour_search_events(G.dev(px), G.dev(py), G.dev(t), W, H, window,
                                        half_extent=half_extent)
    assert csr.nnz == len(ci)
    assert np.array_equal(csr.row_ptr.cpu().numpy(), rp)
    assert np.array_equal(csr.col_idx[:csr.nnz].cpu().numpy(), ci)
    check_events_csc(px, py, t, W, H, window, half_extent, rp, ci)


def check_events_csc(px, py, t, W, H, window, half_extent, rp, ci):
    """The combined search gives the same CSR and, as its CSC, the oracle's
    reverse pattern (the same entries as the transpose, columns in block
    order), bit-exact."""
    csr, csc = G.sbc.neighbour_search_events_csc(G.dev(px), G.dev(py), G.dev(t), W, H, window,
                                                 half_extent=half_extent)
    assert csr.nnz == len(ci) and csc.edge_perm is None
    assert np.array_equal(csr.row_ptr.cpu().numpy(), rp)
    assert np.array_equal(csr.col_idx[:csr.nnz].cpu().numpy(), ci)
    cp, ri = oracle.events_csc(px, py, t, window, half_extent, W, H)
    assert np.array_equal(csc.col_ptr.cpu().numpy(), cp)
    assert np.array_equal(csc.row_idx[:len(ci)].cpu().numpy(), ri)


EVENT_CASES = ["ev_small", "ev_odd", "fz_ev32", "fz_tiny_ev", "events_300k", "events_1m_bf16"]


@pytest.mark.parametrize("name", EVENT_CASES)
def test_events_csc_bit_exact(name):
    print(f"[events csc] {name}", flush=True)
    w, rp, ci, _ = case(name)
    check_events_csc(w["px"], w["py"], w["t"], w["width"], w["height"], w["window"],
                     w.get("half_extent", 1), rp, ci)


@pytest.mark.parametrize("window", [0, 7, 2**31 - 1])
def test_events_csc_window_edges(window):
    """Equal timestamps, gaps of exactly the window, and timestamps near the
    int32 limits with a window that would overflow t + window."""
    print(f"[events csc window] {window}", flush=True)
    rng = np.random.default_rng(window % 1000)
    n, W, H = 3000, 6, 5
    px = rng.integers(0, W, size=n).astype(np.int32)
    py = rng.integers(0, H, size=n).astype(np.int32)
    steps = rng.choice([0, 0, 7, 1, 8], size=n)
    t = (np.cumsum(steps) + (2**31 - 1 - steps.sum() if window > 1000 else 0)).astype(np.int64)
    t = t.astype(np.int32)
    rp, ci = oracle.events_csr(px, py, t, window, 1, W, H)
    check_events_csc(px, py, t, W, H, window, 1, rp, ci)


@pytest.mark.parametrize("order", ORDERS)
@pytest.mark.parametrize("name", ["ev_small", "ev_bf16", "fz_ev32", "fz_tiny_ev", "pts_down",
                                  "fz_pts64", "pts_mono4_odd"])
def test_backward_without_edge_perm(name, order):
    """With the basis evaluated inside, a CSC without edge_perm gives the same
    gradients, bit for bit, on the fused and the separate-kernel routes (the
    values of the transposed entries are then evaluated in their own order).
    For an event stream, the CSC of the search itself (its columns in block
    order, so another order of the same sums) gives them within the case's
    tolerance."""
    print(f"[backward no perm] {name} {order}", flush=True)
    w, rp, ci, v = case(name)
    t, csr = gpu_case(name)
    geo = G.geometry(w, t)
    csc = G.sbc.csr_transpose(csr)
    dF, dW = G.sbc.conv_backward(csr, csc, t["F"], t["W"], t["dY"], geometry=geo, order=order)
    bare = G.sbc.CSC(csc.col_ptr, csc.row_idx, None, csc.n_cols)
    dF2, dW2 = G.sbc.conv_backward(csr, bare, t["F"], t["W"], t["dY"], geometry=geo, order=order)
    assert np.array_equal(dF2.cpu().numpy(), dF.cpu().numpy())
    assert np.array_equal(dW2.cpu().numpy(), dW.cpu().numpy())
    if w["kind"] == "events":
        csr2, found = G.sbc.neighbour_search_events_csc(t["px"], t["py"], t["t"], w["width"],
                                                        w["height"], w["window"])
        assert np.array_equal(csr2.col_idx[:csr2.nnz].cpu().numpy(), ci)
        dF3, dW3 = G.sbc.conv_backward(csr, found, t["F"], t["W"], t["dY"], geometry=geo,
                                       order=order)
        assert G.row_error(dF3.cpu().numpy(), dF.cpu().numpy()) < tol(w)
        assert G.norm_error(dW3.cpu().numpy(), dW.cpu().numpy()) < tol(w)
    vv = G.sbc.basis_eval(csr, geo)
    with pytest.raises(G.sbc.ops.L.SbcError, match="INVALID_ARG"):
        G.sbc.conv_backward(csr, bare, t["F"], t["W"], t["dY"], v=vv, order=order)


@pytest.mark.parametrize("name", ["ev_small", "ev_bf16", "fz_ev32", "fz_tiny_ev"])
def test_event_backward_wide_offset_path(name, monkeypatch):
    """The fixed-decay event backward takes the generic gather (64-bit
    addressing) when its arrays pass 4 GiB; the environment variable
    SBC_EVENT8_WIDE_PATH=1 takes it at any size.  Both paths agree with the
    oracle."""
    print(f"[backward wide path] {name}", flush=True)
    w, rp, ci, v = case(name)
    t, csr = gpu_case(name)
    csc = G.sbc.csr_transpose(csr)
    dF_ref, dW_ref = oracle_backward(name)
    monkeypatch.setenv("SBC_EVENT8_WIDE_PATH", "1")
    dF, dW = G.sbc.conv_backward(csr, csc, t["F"], t["W"], t["dY"], geometry=G.geometry(w, t),
                                 order="spmm_first")
    monkeypatch.delenv("SBC_EVENT8_WIDE_PATH")
    assert G.row_error(dF.cpu().numpy(), dF_ref) < tol(w)
    assert G.norm_error(dW.cpu().numpy(), dW_ref) < tol(w)


@pytest.mark.parametrize("name", ["fz_ev32", "fz_tiny_ev", "events_300k"])
def test_event_forward_one_hot_path(name, monkeypatch):
    """The fixed-decay event forward on rows of 32 float32 channels keeps each
    lane's G values for all offsets in LDS and adds an edge into its offset's
    only; with SBC_EVENT8_WIDE_PATH=1 (or arrays past 4 GiB) it takes the
    register forward, which multiplies all offsets.  Both take the edges of a
    (row, offset, channel) sum in pattern order and contract G W in the same
    order, so they agree exactly, and with the oracle."""
    print(f"[forward one-hot path] {name}", flush=True)
    w, rp, ci, v = case(name)
    assert w["C_in"] == 32 and w["C_out"] == 32 and w["dtype"] == "f32"
    t, csr = gpu_case(name)
    Y = G.sbc.conv_forward(csr, t["F"], t["W"], geometry=G.geometry(w, t), order="spmm_first")
    monkeypatch.setenv("SBC_EVENT8_WIDE_PATH", "1")
    Y_reg = G.sbc.conv_forward(csr, t["F"], t["W"], geometry=G.geometry(w, t), order="spmm_first")
    monkeypatch.delenv("SBC_EVENT8_WIDE_PATH")
    Y, Y_reg = Y.cpu().numpy(), Y_reg.cpu().numpy()
    assert np.array_equal(Y, Y_reg)
    assert G.row_error(Y, oracle_forward(name)) < tol(w)


def test_transpose_by_radix_sort():
    """Patterns of 2^21 edges or more are transposed by the radix sort; trailing
    columns without edges must still get their (empty) ranges."""
    rng = np.random.default_rng(77)
    n_rows, n_cols = 300_000, 160_000
    lens = rng.integers(4, 11, size=n_rows)
    rp = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    assert rp[-1] >= 1 << 21
    # columns drawn from the first 120k only: the last 40k columns stay empty
    starts = rng.integers(0, 120_000 - 12, size=n_rows)
    ci = np.concatenate([s + np.sort(rng.choice(12, size=k, replace=False))
                         for s, k in zip(starts, lens)]).astype(np.int32)
    csr = G.sbc.CSR(G.dev(rp), G.dev(ci), n_rows, n_cols, len(ci))
    csc = G.sbc.csr_transpose(csr)
    cp, ri, perm = oracle.csr_transpose(rp, ci, n_cols)
    assert np.array_equal(csc.col_ptr.cpu().numpy(), cp)
    assert np.array_equal(csc.row_idx[:len(ci)].cpu().numpy(), ri)
    assert np.array_equal(csc.edge_perm[:len(ci)].cpu().numpy(), perm)


# ---------------------------------------------------------------- featureless convolution
@pytest.mark.parametrize("materialised", [False, True])
@pytest.mark.parametrize("name", ["pts_weighted", "pts_down", "pts_mono4_odd", "ev_small",
                                  "pts_weighted_odd", "ellipsoids_featureless"])
def test_featureless(name, materialised):
    """Z = G~ Phi_0 and dPhi_0 = G~^T dZ (Eq. 9-10) against the oracle, with the
    basis evaluated inside or read from v; Phi_0 is W[:, 0, :], dZ is dY."""
    print(f"[featureless] {name} materialised={materialised}", flush=True)
    w, rp, ci, v = case(name)
    t, csr = gpu_case(name)
    Phi = np.ascontiguousarray(np.asarray(w["W"], np.float32)[:, 0, :])
    dZ = np.asarray(w["dY"], np.float32)
    Z_ref, _ = oracle.conv.featureless_forward(rp, ci, v, Phi)
    dPhi_ref = oracle.conv.featureless_backward(rp, ci, v, dZ)
    geo = G.geometry(w, t)
    vv = G.sbc.basis_eval(csr, geo) if materialised else None
    kw = dict(v=vv) if materialised else dict(geometry=geo)
    Z = G.sbc.featureless_forward(csr, G.dev(Phi), **kw).cpu().numpy()
    dPhi = G.sbc.featureless_backward(csr, G.dev(dZ), w["M"], **kw).cpu().numpy()
    e1 = G.row_error(Z, Z_ref)
    e2 = G.norm_error(dPhi, dPhi_ref)
    print(f"    Z row error {e1:.3e}  dPhi error {e2:.3e}", flush=True)
    assert e1 < G.TOL_F32 and e2 < G.TOL_F32
    empty = np.nonzero(np.diff(rp) == 0)[0]
    assert np.all(Z[empty] == 0)


# ---------------------------------------------------------------- up-sampling shapes
def _upsampling_case():
    """Inputs are a quarter of each cloud, outputs the whole cloud, and the
    channels shrink (48 -> 16): the up-sampling convolution of Table 1."""
    rng = np.random.default_rng(21)
    clouds = []
    for b in range(3):
        x = workloads.ellipsoid_surface_points(rng, 400 + 31 * b, rng.uniform(0.5, 1.0, size=3))
        clouds.append((x[: len(x) // 4], x))
    w = workloads.points_workload(rng, clouds, workloads.BASIS_MONO8, 0.3, 0, 48, 16)
    rp, ci = oracle.points_csr(w["x_in"], w["in_splits"], w["x_out"], w["out_splits"],
                               w["radius"], 0)
    v = oracle.basis.point_values(w["basis"], w["x_in"], w["x_out"], rp, ci, w["radius"], w["M"])
    return w, rp, ci, v


@pytest.mark.parametrize("order", ["auto"] + ORDERS)
def test_upsampling(order):
    print(f"[upsampling] {order}", flush=True)
    w, rp, ci, v = _upsampling_case()
    assert w["n_out"] > w["n_in"] and w["C_in"] > w["C_out"]
    t = G.to_device(w)
    csr = G.search(w, t)
    assert np.array_equal(csr.col_idx[:csr.nnz].cpu().numpy(), ci)
    plan = G.sbc.conv_plan(w["n_out"], w["n_in"], csr.nnz, w["M"], w["C_in"], w["C_out"])
    assert plan["forward_order"] == "gemm_first"     # Table 1: N (F W) for up-sampling
    geo = G.geometry(w, t)
    Y = G.sbc.conv_forward(csr, t["F"], t["W"], geometry=geo, order=order).cpu().numpy()
    assert G.row_error(Y, oracle.conv.forward(rp, ci, v, w["F"], w["W"])) < G.TOL_F32
    csc = G.sbc.csr_transpose(csr)
    dF, dW = G.sbc.conv_backward(csr, csc, t["F"], t["W"], t["dY"], geometry=geo, order=order)
    dF_ref, dW_ref = oracle.conv.backward(rp, ci, v, w["F"], w["W"], w["dY"], w["n_in"])
    assert G.row_error(dF.cpu().numpy(), dF_ref) < G.TOL_F32
    assert G.norm_error(dW.cpu().numpy(), dW_ref) < G.TOL_F32


# ---------------------------------------------------------------- learned decay rates
@pytest.mark.parametrize("route", ["sparse_product", "fused"])
@pytest.mark.parametrize("name", ["ev_decays2", "ev_decays3_odd", "ev_decays4_bf16",
                                  "fz_ev_decays2_32", "events_300k_decays2"])
def test_decay_gradient(name, route):
    """d<Y, dY>/d lambda of the learned-decay kernel (Eq. 12) against the oracle's
    per-edge chain rule: without the transpose (G' = N' F route), and with the
    transpose from the reverse search (the fused D-route where the shape has one)."""
    print(f"[decay gradient] {name} {route}", flush=True)
    w, rp, ci, v = case(name)
    t, csr = gpu_case(name)
    csc = None
    if route == "fused":
        _, csc = G.sbc.neighbour_search_events_csc(t["px"], t["py"], t["t"], w["width"],
                                                   w["height"], w["window"])
    dl = G.sbc.conv_decay_gradient(csr, t["F"], t["W"], t["dY"], G.geometry(w, t),
                                   csc=csc).cpu().numpy()
    vd = oracle.basis.event_decay_basis(w["px"], w["py"], w["t"], rp, ci, w["decays"],
                                        derivative=True)
    ref = oracle.conv.decay_backward(rp, ci, vd, w["F"], w["W"], w["dY"])
    err = G.norm_error(dl, ref)
    print(f"    dlambda error {err:.3e}", flush=True)
    assert err < tol(w)


@pytest.mark.parametrize("name", ["fz_ev_decays2_32", "events_300k_decays2"])
def test_decay_backward_wide_offset_path(name, monkeypatch):
    """The learned-decay backward and decay gradient on rows of 32 float32
    channels take the in-place gather (32-bit byte offsets); past 4 GiB, or
    with SBC_EVENT8_WIDE_PATH=1, the generic gather.  Both paths agree with
    the oracle."""
    print(f"[decay wide path] {name}", flush=True)
    w, rp, ci, v = case(name)
    assert w["C_in"] == 32 and w["C_out"] == 32 and w["dtype"] == "f32"
    t, csr = gpu_case(name)
    csc = G.sbc.csr_transpose(csr)
    dF_ref, dW_ref = oracle_backward(name)
    vd = oracle.basis.event_decay_basis(w["px"], w["py"], w["t"], rp, ci, w["decays"],
                                        derivative=True)
    dl_ref = oracle.conv.decay_backward(rp, ci, vd, w["F"], w["W"], w["dY"])
    for wide in (False, True):
        if wide:
            monkeypatch.setenv("SBC_EVENT8_WIDE_PATH", "1")
        dF, dW = G.sbc.conv_backward(csr, csc, t["F"], t["W"], t["dY"],
                                     geometry=G.geometry(w, t), order="spmm_first")
        dl = G.sbc.conv_decay_gradient(csr, t["F"], t["W"], t["dY"], G.geometry(w, t),
                                       csc=csc).cpu().numpy()
        monkeypatch.delenv("SBC_EVENT8_WIDE_PATH", raising=False)
        assert G.row_error(dF.cpu().numpy(), dF_ref) < tol(w)
        assert G.norm_error(dW.cpu().numpy(), dW_ref) < tol(w)
        assert G.norm_error(dl, dl_ref) < tol(w)


# ---------------------------------------------------------------- subsampling
def _sampling_batch(seed, sizes, doubled=False):
    """Ellipsoid clouds; doubled: each cloud is sizes[b] / 2 distinct points
    followed by a copy of each (coincident points)."""
    rng = np.random.default_rng(seed)
    xs = []
    for n in sizes:
        m = n // 2 if doubled else n
        c = (workloads.ellipsoid_surface_points(rng, m, rng.uniform(0.5, 1.0, size=3))
             if m else np.zeros((0, 3)))
        xs.append(np.concatenate([c, c]) if doubled else c)
    x = np.concatenate(xs).astype(np.float32)
    return x, np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)


# (seed, cloud sizes, ball radius, points per cloud[, doubled])
SAMPLING_CASES = {"small": (30, [300, 0, 1, 450], 0.2, 100),
                  "c2_clouds": (31, [1024] * 32, 0.1, 256),
                  "large_cloud": (32, [8192, 700], 0.05, 2000),
                  "coincident_whole_clouds": (33, [80, 600, 2], 0.15, 600, True)}


@pytest.mark.parametrize("method", ["ifp", "approx_ifp", "rejection", "approx_ifp_rejection"])
@pytest.mark.parametrize("case_name", list(SAMPLING_CASES))
def test_sampling_bit_exact(case_name, method):
    """Indices, bounds and squared distances equal the oracle's exactly."""
    print(f"[sampling] {case_name} {method}", flush=True)
    seed, sizes, radius, per, *doubled = SAMPLING_CASES[case_name]
    x, splits = _sampling_batch(seed, sizes, bool(doubled))
    rp, ci = oracle.points_csr(x, splits, x, splits, radius, 0)
    xd, sd = G.dev(x), G.dev(splits)
    ball = G.sbc.neighbour_search_points(xd, sd, xd, sd, radius, 0)
    idx, osp, d2 = G.sbc.sample_points(xd, sd, method, per, ball=ball, with_dmin=True)
    if method == "ifp":
        ref, dref = oracle.sampling.ifp(x, splits, [min(per, n) for n in sizes])
    elif method == "approx_ifp":
        ref, dref = oracle.sampling.approx_ifp(x, splits, [min(per, n) for n in sizes], rp, ci)
    elif method == "rejection":
        taken, dref = oracle.sampling.rejection_sampling(x, splits, rp, ci)
        ref = np.nonzero(taken)[0].astype(np.int32)
    else:
        ref, dref = oracle.sampling.approx_ifp_after_rejection(x, splits, per, rp, ci)
    osp = osp.cpu().numpy()
    assert osp[-1] == len(ref)
    assert np.array_equal(idx.cpu().numpy()[:len(ref)], ref)
    assert np.array_equal(d2.cpu().numpy()[:len(x)], dref)
    if method == "rejection":
        want = np.searchsorted(ref, splits)      # taken points per cloud, in order
        assert np.array_equal(osp, want)
    elif doubled:                                # whole clouds: every point once
        assert sorted(ref.tolist()) == list(range(len(x)))


# ---------------------------------------------------------------- LIF event sampler
# (seed, n, width, height, duration, kernel, stride, decay, thresh, reset)
LIF_CASES = {
    "nmnist_k3s2": (40, 5000, 34, 34, 30_000, 3, 2, 2000.0, 1.5, -3.0),
    "k5s1": (41, 4000, 23, 17, 20_000, 5, 1, 1000.0, 1.25, -2.0),
    "k4s2_even": (42, 4000, 19, 21, 20_000, 4, 2, 1500.0, 1.0, -3.0),
    "k1s2_unreached": (43, 3000, 15, 9, 10_000, 1, 2, 3000.0, 1.5, 0.0),
    "k2s3": (44, 3000, 31, 12, 10_000, 2, 3, 500.0, 0.7, 0.1),
}


def _lif_ref(px, py, t, W, H, k, S, decay, th, rs):
    out = oracle.sampling.lif(px, py, t, W, H, k, S, decay, th, rs)
    return out[:, 1].astype(np.int32), out[:, 2].astype(np.int32), t[out[:, 0]], \
        out[:, 0].astype(np.int32)


def _lif_check(px, py, t, W, H, k, S, decay, th, rs):
    x, y, tt, src, cnt = G.sbc.lif_sample_events(G.dev(px), G.dev(py), G.dev(t), W, H, k, S,
                                                 decay, th, rs)
    rx, ry, rt, rsrc = _lif_ref(px, py, t, W, H, k, S, decay, th, rs)
    print(f"    {len(px)} events -> {cnt} (oracle {len(rx)})", flush=True)
    assert cnt == len(rx)
    for a, b in [(src, rsrc), (x, rx), (y, ry), (tt, rt)]:
        assert np.array_equal(a.cpu().numpy(), b)
    return cnt


@pytest.mark.parametrize("case_name", list(LIF_CASES))
def test_lif_bit_exact(case_name):
    """Output events (cell, time, source event), in emission order, equal the
    oracle's exactly."""
    print(f"[lif] {case_name}", flush=True)
    seed, n, W, H, dur, k, S, decay, th, rs = LIF_CASES[case_name]
    px, py, t, _ = workloads.uniform_events(np.random.default_rng(seed), n, W, H, dur)
    assert _lif_check(px, py, t, W, H, k, S, decay, th, rs) > 0


def test_lif_full_size_workload():
    """The benchmarked stream (300k events on 128 x 128, 3 x 3 fields, stride
    2, the CIFAR10-DVS settings), every output event against the oracle."""
    print("[lif] events_300k_lif", flush=True)
    w = workloads.events_300k_lif()
    assert _lif_check(w["px"], w["py"], w["t"], w["width"], w["height"], w["kernel"],
                      w["stride"], w["decay"], w["v_thresh"], w["v_reset"]) > 10_000


def test_lif_exact_ties_and_bursts():
    """No decay, equal times and thresholds the potentials reach exactly
    (multiples of 1/4 and 1/2): the comparison is strict on both sides.  Also a
    bursty stream with a long decay (many spikes per cell)."""
    print("[lif] ties", flush=True)
    rng = np.random.default_rng(46)
    n = 6000
    px = rng.integers(0, 8, n).astype(np.int32)
    py = rng.integers(0, 8, n).astype(np.int32)
    t = np.sort(rng.integers(0, 50, n)).astype(np.int32)
    _lif_check(px, py, t, 8, 8, 3, 2, np.inf, 1.0, 0.0)
    _lif_check(px, py, t, 8, 8, 3, 2, 1e12, 1.5, -0.5)
    px, py, t, _ = workloads.bursty_events(rng, 20_000, 40, 30, 40_000)
    _lif_check(px, py, t, 40, 30, 3, 2, 20_000.0, 1.5, -2.0)


def test_lif_crowded_cells():
    """Cells whose receptive field holds more events than the LDS staging (a
    hot pixel, and a tiny sensor) take the one-lane path; the rest of the grid
    the wave path; both equal the oracle."""
    print("[lif] crowded", flush=True)
    rng = np.random.default_rng(48)
    n = 12_000
    px = rng.integers(0, 30, n).astype(np.int32)
    py = rng.integers(0, 20, n).astype(np.int32)
    hot = rng.random(n) < 0.25
    px[hot], py[hot] = 5, 5
    t = np.sort(rng.integers(0, 60_000, n)).astype(np.int32)
    _lif_check(px, py, t, 30, 20, 3, 2, 2000.0, 1.5, -3.0)
    px, py, t, _ = workloads.uniform_events(rng, 20_000, 4, 4, 50_000)
    _lif_check(px, py, t, 4, 4, 3, 2, 2000.0, 1.5, -3.0)
    _lif_check(px, py, t, 4, 4, 5, 1, 500.0, 1.2, -1.0)


def test_lif_empty_and_capacity():
    """An empty stream gives no events; a capacity below the count keeps the
    first events and, when synchronised, reports the shortfall; without
    synchronisation the device count is exact."""
    print("[lif] empty / capacity", flush=True)
    e = G.dev(np.zeros(0, np.int32))
    assert G.sbc.lif_sample_events(e, e, e, 10, 10)[4] == 0
    seed, n, W, H, dur, k, S, decay, th, rs = LIF_CASES["nmnist_k3s2"]
    px, py, t, _ = workloads.uniform_events(np.random.default_rng(seed), n, W, H, dur)
    rx, ry, rt, rsrc = _lif_ref(px, py, t, W, H, k, S, decay, th, rs)
    args = (G.dev(px), G.dev(py), G.dev(t), W, H, k, S, decay, th, rs)
    with pytest.raises(G.sbc.ops.L.SbcError, match="capacity"):
        G.sbc.lif_sample_events(*args, capacity=len(rx) - 1)
    x, y, tt, src, cnt = G.sbc.lif_sample_events(*args, capacity=100, sync=False)
    assert int(cnt.item()) == len(rx)
    assert np.array_equal(src[:100].cpu().numpy(), rsrc[:100])
    assert np.array_equal(x[:100].cpu().numpy(), rx[:100])


def test_lif_rejects_bad_streams():
    """Pixels off the sensor and decreasing times are reported (synchronised
    calls); kernel sizes past 5 are refused before any launch."""
    print("[lif] errors", flush=True)
    px = G.dev(np.array([0, 1, 40], np.int32))
    py = G.dev(np.array([0, 1, 2], np.int32))
    t = G.dev(np.array([0, 5, 9], np.int32))
    with pytest.raises(G.sbc.ops.L.SbcError, match="outside"):
        G.sbc.lif_sample_events(px, py, t, 10, 10)
    px = G.dev(np.array([0, 1, 2], np.int32))
    with pytest.raises(G.sbc.ops.L.SbcError, match="non-decreasing"):
        G.sbc.lif_sample_events(px, py, G.dev(np.array([0, 9, 5], np.int32)), 10, 10)
    with pytest.raises(G.sbc.ops.L.SbcError, match="kernel"):
        G.sbc.lif_sample_events(px, py, t, 10, 10, kernel=6)


# ---------------------------------------------------------------- deployment stream
@pytest.mark.parametrize("pieces,P", [([3000], 10), ([1, 699, 0, 1, 1299, 1000], 10),
                                      ([1, 1500, 1499], 136)])
def test_event_stream_matches_the_recursion(pieces, P):
    """The stream fed in batches (the state carried on the device) gives the
    outputs and final state of the oracle's per-event recursion over the whole
    stream, within 1e-5 (row-normwise; the state is float32 and the batch sums
    come in another order); the last-update times are exact.  Channel counts
    that are not multiples of 4, C_in != C_out, and a wide output (136)."""
    print(f"[stream] pieces {pieces} P {P}", flush=True)
    rng = np.random.default_rng(50)
    n, Wd, H, tau = 3000, 20, 16, 3000.0
    px, py, t, _ = workloads.uniform_events(rng, n, Wd, H, 30_000)
    F = rng.standard_normal((n, 6)).astype(np.float32)
    W = (rng.standard_normal((8, 6, P)) / np.sqrt(48)).astype(np.float32)
    Y_ref, z_ref, last_ref = oracle.conv.deployment_stream(px, py, t, F.astype(np.float64),
                                                           W.astype(np.float64), Wd, H, tau)
    st = G.sbc.EventStream(Wd, H, 6, tau, device=G.DEV)
    Wd_dev = G.dev(W)
    Ys, a = [], 0
    for k in pieces:
        b = a + k
        Ys.append(st.step(G.dev(px[a:b]), G.dev(py[a:b]), G.dev(t[a:b]), G.dev(F[a:b]), Wd_dev)
                  .cpu().numpy())
        a = b
    assert a == n
    Y = np.concatenate(Ys)
    err = G.row_error(Y, Y_ref)
    zerr = G.row_error(st.z.cpu().numpy(), z_ref.reshape(Wd * H, 6))
    print(f"    Y {err:.2e}  z {zerr:.2e}", flush=True)
    assert err < 1e-5 and zerr < 1e-5
    assert np.array_equal(st.z_time.cpu().numpy(), last_ref.reshape(-1).astype(np.int32))


@pytest.mark.parametrize("Mv,C_in,pieces", [(1, 10, [4000]), (2, 6, [1, 1999, 0, 2000]),
                                             (3, 5, [700, 3300]), (4, 10, [2500, 1500])])
def test_event_stream_learned_decays(Mv, C_in, pieces):
    """The deployment form with learned decays (M_v rates per offset, a state
    per basis function) fed in batches against the oracle's recursion over
    the whole stream: outputs and final state within 1e-5, times exact.  Ten
    input channels give three 4-channel chunks per state, so one pixel's
    threads straddle waves."""
    print(f"[stream] decays Mv {Mv} C_in {C_in} pieces {pieces}", flush=True)
    rng = np.random.default_rng(52 + Mv)
    n, Wd, H, P = 4000, 18, 14, 12
    px, py, t, _ = workloads.uniform_events(rng, n, Wd, H, 40_000)
    lam = rng.uniform(1 / 20_000, 1 / 500, (8, Mv)).astype(np.float32)
    F = rng.standard_normal((n, C_in)).astype(np.float32)
    W = (rng.standard_normal((8 * Mv, C_in, P)) / np.sqrt(8 * Mv * C_in)).astype(np.float32)
    Y_ref, z_ref, last_ref = oracle.conv.deployment_stream(
        px, py, t, F.astype(np.float64), W.astype(np.float64), Wd, H, None,
        decays=lam.astype(np.float64))
    st = G.sbc.EventStream(Wd, H, C_in, device=G.DEV, decays=G.dev(lam))
    Wdev = G.dev(W)
    Ys, a = [], 0
    for k in pieces:
        b = a + k
        Ys.append(st.step(G.dev(px[a:b]), G.dev(py[a:b]), G.dev(t[a:b]), G.dev(F[a:b]), Wdev)
                  .cpu().numpy())
        a = b
    assert a == n
    err = G.row_error(np.concatenate(Ys), Y_ref)
    zerr = G.row_error(st.z.cpu().numpy().reshape(-1, C_in), z_ref.reshape(-1, C_in))
    print(f"    Y {err:.2e}  z {zerr:.2e}", flush=True)
    assert err < 1e-5 and zerr < 1e-5
    assert np.array_equal(st.z_time.cpu().numpy(), last_ref.reshape(-1).astype(np.int32))


def test_event_stream_wide_fixed_decay_state():
    """The fixed-decay form with ten input channels (three chunks a pixel, a
    pixel's threads in two waves) and one batch: times and state exact to
    the recursion within 1e-5."""
    print("[stream] fixed decay C_in 10", flush=True)
    rng = np.random.default_rng(56)
    n, Wd, H, tau = 3000, 12, 10, 4000.0
    px, py, t, _ = workloads.uniform_events(rng, n, Wd, H, 30_000)
    F = rng.standard_normal((n, 10)).astype(np.float32)
    W = (rng.standard_normal((8, 10, 4)) / 9).astype(np.float32)
    Y_ref, z_ref, last_ref = oracle.conv.deployment_stream(px, py, t, F.astype(np.float64),
                                                           W.astype(np.float64), Wd, H, tau)
    st = G.sbc.EventStream(Wd, H, 10, tau, device=G.DEV)
    Y = st.step(G.dev(px), G.dev(py), G.dev(t), G.dev(F), G.dev(W)).cpu().numpy()
    err = G.row_error(Y, Y_ref)
    zerr = G.row_error(st.z.cpu().numpy(), z_ref.reshape(-1, 10))
    print(f"    Y {err:.2e}  z {zerr:.2e}", flush=True)
    assert err < 1e-5 and zerr < 1e-5
    assert np.array_equal(st.z_time.cpu().numpy(), last_ref.reshape(-1).astype(np.int32))


def test_event_stream_decays_rejects_bad_arguments():
    """Rates of the wrong shape, too many decays and a mismatched W are refused."""
    print("[stream] decays refusals", flush=True)
    with pytest.raises(ValueError, match="M_v"):
        G.sbc.EventStream(8, 8, 4, device=G.DEV, decays=G.dev(np.ones((8, 5), np.float32)))
    with pytest.raises(ValueError, match="tau"):
        G.sbc.EventStream(8, 8, 4, device=G.DEV)
    st = G.sbc.EventStream(8, 8, 4, device=G.DEV, decays=G.dev(np.ones((8, 2), np.float32)))
    e = G.dev(np.zeros(3, np.int32))
    with pytest.raises(ValueError, match="16"):
        st.step(e, e, e, G.dev(np.zeros((3, 4), np.float32)),
                G.dev(np.zeros((8, 4, 2), np.float32)))


def test_event_stream_full_size_batches():
    """The benchmarked form: the 300k-event stream (128 x 128, 32 -> 32
    channels, tau 10 ms) in batches of 4096; sampled outputs of the last batch
    and the final state against the oracle's recursion over the whole stream."""
    print("[stream] events_stream", flush=True)
    w = workloads.events_stream()
    n, B = w["n_in"], w["batch"]
    Y_ref, z_ref, last_ref = oracle.conv.deployment_stream(
        w["px"], w["py"], w["t"], w["F"].astype(np.float64), w["W"].astype(np.float64),
        w["width"], w["height"], w["tau"])
    st = G.sbc.EventStream(w["width"], w["height"], w["C_in"], w["tau"], device=G.DEV)
    t = G.to_device(w)
    Wdev = t["W"]
    for a in range(0, n, B):
        Y = st.step(t["px"][a:a + B], t["py"][a:a + B], t["t"][a:a + B], t["F"][a:a + B], Wdev)
    last = Y.cpu().numpy()
    a = (n - 1) // B * B
    err = G.row_error(last, Y_ref[a:])
    zerr = G.row_error(st.z.cpu().numpy(), z_ref.reshape(-1, w["C_in"]))
    print(f"    Y {err:.2e}  z {zerr:.2e}", flush=True)
    assert err < 1e-5 and zerr < 1e-5
    assert np.array_equal(st.z_time.cpu().numpy(), last_ref.reshape(-1).astype(np.int32))


def test_lif_bursty_1m_stream():
    """The 1M-event bursty stream on 346 x 260 (a 173 x 130 grid, 3 x 3 fields,
    stride 2) with the N-Caltech101 settings of the supplementary's table
    (decay 1 ms, threshold 1.25, reset -2): every output event against the
    oracle."""
    print("[lif] bursty 1M", flush=True)
    w = workloads.bursty_event_stream()
    assert _lif_check(w["px"], w["py"], w["t"], w["width"], w["height"], 3, 2, 1000.0, 1.25,
                      -2.0) > 10_000
