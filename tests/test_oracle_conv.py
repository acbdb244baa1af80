"""Pins of the oracle's forward and backward (CPU only).

The oracle evaluates the convolution edge by edge (the finite sum with the
basis kernel).  These tests check it against hand-computed cases, the
method's matrix form evaluated with dense matrices, a textbook 2D convolution,
the event convolution's deployment recursion, invariances, adjoint identities
and finite differences.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
import workloads
from oracle.basis import event_basis, event_offset_index, point_basis

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def _points_problem(w):
    rp, ci = oracle.points_csr(w["x_in"], w["in_splits"], w["x_out"], w["out_splits"],
                               w["radius"], w["k_cap"])
    v = point_basis(w["x_in"], w["x_out"], rp, ci, w["radius"], w["M"])
    return rp, ci, v


def _events_problem(w):
    rp, ci = oracle.events_csr(w["px"], w["py"], w["t"], w["window"], 1, w["width"], w["height"])
    v = event_basis(w["px"], w["py"], w["t"], rp, ci, w["tau"])
    return rp, ci, v


# ---------------------------------------------------------------- hand cases
def test_points_hand_case():
    g = _gold("points_hand_case.json")
    F, W, dY = (np.array(g[k], np.float64) for k in ("F", "W", "dY"))
    for variant, k_cap in (("uncapped", 0), ("cap2", 2)):
        rp, ci = oracle.points_csr(np.array(g["x_in"], np.float32), np.array([0, 4], np.int32),
                                   np.array(g["x_out"], np.float32), np.array([0, 1], np.int32),
                                   g["radius"], k_cap)
        v = point_basis(np.array(g["x_in"]), np.array(g["x_out"]), rp, ci, g["radius"], 4)
        Y = oracle.conv.forward(rp, ci, v, F, W)
        dF, dW = oracle.conv.backward(rp, ci, v, F, W, dY, 4)
        assert Y.tolist() == g[variant]["Y"]
        assert dF.tolist() == g[variant]["dF"]
        if "dW" in g[variant]:
            assert dW.tolist() == g[variant]["dW"]
    assert g["mirrored_sign_reading_Y"] != g["uncapped"]["Y"][0][0]


def test_events_hand_case():
    g = _gold("events_hand_case.json")
    rp, ci = oracle.events_csr(g["px"], g["py"], g["t"], g["window"], 1, 10, 10)
    v = event_basis(g["px"], g["py"], g["t"], rp, ci, g["tau"])
    W = np.array(g["W_m"], np.float64).reshape(8, 1, 1)
    Y = oracle.conv.forward(rp, ci, v, np.array(g["F"]), W)
    np.testing.assert_allclose(Y[:, 0], g["Y"], rtol=1e-15, atol=0)
    assert Y[0, 0] == 0.0 and Y[4, 0] == 0.0


# ---------------------------------------------------------------- dense form
def _dense_matrices(rp, ci, v, n_in):
    """The M neighbourhood matrices N^(m) as dense arrays."""
    n_out = len(rp) - 1
    A = np.zeros((v.shape[1], n_out, n_in))
    rows = oracle.basis.edge_rows(rp)
    for m in range(v.shape[1]):
        A[m, rows, ci] = v[:, m]
    return A


@pytest.mark.parametrize("kind", ["points", "events"])
def test_dense_matrix_form(kind):
    """sum_m N^(m) F W^(m) with dense matrices (Section 3.1, the matrix-product form)."""
    if kind == "points":
        w = workloads.small_points(seed=1, n=48, n_clouds=2, n_out=20, c_in=5, c_out=7)
        rp, ci, v = _points_problem(w)
    else:
        w = workloads.small_events(seed=2, n=60, width=4, height=3, c=6)
        rp, ci, v = _events_problem(w)
    A = _dense_matrices(rp, ci, v, w["n_in"])
    F, W, dY = (w[k].astype(np.float64) for k in ("F", "W", "dY"))
    Y_dense = sum(A[m] @ F @ W[m] for m in range(w["M"]))
    dF_dense = sum(A[m].T @ dY @ W[m].T for m in range(w["M"]))
    dW_dense = np.stack([(A[m] @ F).T @ dY for m in range(w["M"])])
    Y = oracle.conv.forward(rp, ci, v, F, W)
    dF, dW = oracle.conv.backward(rp, ci, v, F, W, dY, w["n_in"])
    np.testing.assert_allclose(Y, Y_dense, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dF, dF_dense, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dW, dW_dense, rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------- invariants
def test_linearity():
    w = workloads.small_points(seed=2, n_out=30)
    rp, ci, v = _points_problem(w)
    rng = np.random.default_rng(0)
    F1, F2 = rng.standard_normal((2, w["n_in"], w["C_in"]))
    W1, W2 = rng.standard_normal((2, w["M"], w["C_in"], w["C_out"]))
    a, b = 0.75, -1.25
    f = lambda F, W: oracle.conv.forward(rp, ci, v, F, W)
    np.testing.assert_allclose(f(a * F1 + b * F2, W1), a * f(F1, W1) + b * f(F2, W1),
                               rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(f(F1, a * W1 + b * W2), a * f(F1, W1) + b * f(F1, W2),
                               rtol=1e-12, atol=1e-12)


def test_adjoint_identities():
    """<Y(F), dY> = <F, dF> = <W, dW> for the bilinear map (F, W) -> Y."""
    for w, prob in ((workloads.small_points(seed=5, n_out=25), _points_problem),
                    (workloads.small_events(seed=3, n=1500), _events_problem)):
        rp, ci, v = prob(w)
        F, W, dY = (w[k].astype(np.float64) for k in ("F", "W", "dY"))
        Y = oracle.conv.forward(rp, ci, v, F, W)
        dF, dW = oracle.conv.backward(rp, ci, v, F, W, dY, w["n_in"])
        s = np.sum(Y * dY)
        assert abs(np.sum(F * dF) - s) <= 1e-10 * max(1.0, abs(s))
        assert abs(np.sum(W * dW) - s) <= 1e-10 * max(1.0, abs(s))


def test_finite_differences():
    """dF and dW are the gradients of <Y, dY> (central differences, exact for a bilinear map)."""
    w = workloads.small_points(seed=6, n=40, n_clouds=1, n_out=12, c_in=3, c_out=4)
    rp, ci, v = _points_problem(w)
    F, W, dY = (w[k].astype(np.float64) for k in ("F", "W", "dY"))
    L = lambda F_, W_: np.sum(oracle.conv.forward(rp, ci, v, F_, W_) * dY)
    dF, dW = oracle.conv.backward(rp, ci, v, F, W, dY, w["n_in"])
    h = 0.5
    for idx in [(0, 0), (3, 2), (17, 1), (39, 0)]:
        E = np.zeros_like(F)
        E[idx] = h
        assert abs((L(F + E, W) - L(F - E, W)) / (2 * h) - dF[idx]) < 1e-12
    for idx in [(0, 0, 0), (7, 2, 3), (4, 1, 1)]:
        E = np.zeros_like(W)
        E[idx] = h
        assert abs((L(F, W + E) - L(F, W - E)) / (2 * h) - dW[idx]) < 1e-12


def test_translation_invariance_points():
    rng = np.random.default_rng(3)
    q = rng.integers(-3000, 3001, size=(400, 3)) / 4096.0
    x = q.astype(np.float32)
    xs = (q + 0.5).astype(np.float32)
    w = workloads.small_points(seed=0, n=400, n_clouds=1)
    F, W = w["F"].astype(np.float64), w["W"].astype(np.float64)
    out = []
    for pts in (x, xs):
        splits = np.array([0, 400], np.int32)
        rp, ci = oracle.points_csr(pts, splits, pts[:150], np.array([0, 150], np.int32), 0.2, 10)
        v = point_basis(pts, pts[:150], rp, ci, 0.2, 8)
        out.append((rp, ci, oracle.conv.forward(rp, ci, v, F, W)))
    assert np.array_equal(out[0][0], out[1][0]) and np.array_equal(out[0][1], out[1][1])
    np.testing.assert_allclose(out[0][2], out[1][2], rtol=1e-12, atol=1e-12)


def test_translation_invariance_events():
    w = workloads.small_events(seed=4)
    rp, ci, v = _events_problem(w)
    t2 = w["t"] + 12345
    rp2, ci2 = oracle.events_csr(w["px"], w["py"], t2, w["window"], 1, w["width"], w["height"])
    v2 = event_basis(w["px"], w["py"], t2, rp2, ci2, w["tau"])
    assert np.array_equal(rp, rp2) and np.array_equal(ci, ci2)
    Y1 = oracle.conv.forward(rp, ci, v, w["F"], w["W"])
    Y2 = oracle.conv.forward(rp2, ci2, v2, w["F"], w["W"])
    np.testing.assert_allclose(Y1, Y2, rtol=1e-13, atol=1e-13)


def test_isolated_outputs_are_exact_zero():
    w = workloads.small_points(seed=8, n_out=10, n_clouds=1)
    x_out = np.concatenate([w["x_out"], np.array([[10, 10, 10]], np.float32)])
    splits_out = np.array([0, len(x_out)], np.int32)
    rp, ci = oracle.points_csr(w["x_in"], w["in_splits"], x_out, splits_out, w["radius"], 0)
    v = point_basis(w["x_in"], x_out, rp, ci, w["radius"], 8)
    Y = oracle.conv.forward(rp, ci, v, w["F"], w["W"])
    assert rp[-1] == rp[-2] and np.all(Y[-1] == 0.0)


def test_permutation_equivariance():
    w = workloads.small_points(seed=9, n_clouds=1, n_out=30)
    perm = np.random.default_rng(1).permutation(w["n_in"])
    x_p = w["x_in"][perm]
    F_p = w["F"][perm]
    rp2, ci2 = oracle.points_csr(x_p, w["in_splits"], w["x_out"], w["out_splits"], w["radius"], 0)
    v2 = point_basis(x_p, w["x_out"], rp2, ci2, w["radius"], 8)
    rp0, ci0 = oracle.points_csr(w["x_in"], w["in_splits"], w["x_out"], w["out_splits"],
                                 w["radius"], 0)
    v0 = point_basis(w["x_in"], w["x_out"], rp0, ci0, w["radius"], 8)
    np.testing.assert_allclose(oracle.conv.forward(rp2, ci2, v2, F_p, w["W"]),
                               oracle.conv.forward(rp0, ci0, v0, w["F"], w["W"]),
                               rtol=1e-12, atol=1e-12)


def test_ragged_batch_is_blockwise():
    w = workloads.small_points(seed=10, n_out=35)
    rp, ci, v = _points_problem(w)
    Y = oracle.conv.forward(rp, ci, v, w["F"], w["W"])
    for b in range(len(w["in_splits"]) - 1):
        i0, i1 = w["in_splits"][b], w["in_splits"][b + 1]
        o0, o1 = w["out_splits"][b], w["out_splits"][b + 1]
        xi, xo = w["x_in"][i0:i1], w["x_out"][o0:o1]
        rb, cb = oracle.points_csr(xi, np.array([0, i1 - i0], np.int32), xo,
                                   np.array([0, o1 - o0], np.int32), w["radius"], w["k_cap"])
        vb = point_basis(xi, xo, rb, cb, w["radius"], 8)
        np.testing.assert_allclose(oracle.conv.forward(rb, cb, vb, w["F"][i0:i1], w["W"]),
                                   Y[o0:o1], rtol=1e-13, atol=1e-13)


def test_sampled_rows_and_columns_match_full():
    w = workloads.small_events(seed=5)
    rp, ci, v = _events_problem(w)
    Y = oracle.conv.forward(rp, ci, v, w["F"], w["W"])
    dF, dW = oracle.conv.backward(rp, ci, v, w["F"], w["W"], w["dY"], w["n_in"])
    rows = np.array([0, 5, 77, w["n_out"] - 1])
    np.testing.assert_array_equal(oracle.conv.forward(rp, ci, v, w["F"], w["W"], rows=rows),
                                  Y[rows])
    dFs, _ = oracle.conv.backward(rp, ci, v, w["F"], w["W"], w["dY"], w["n_in"],
                                  cols_subset=rows, want_dW=False)
    np.testing.assert_allclose(dFs, dF[rows], rtol=1e-14, atol=1e-14)


# ---------------------------------------------------------------- special cases
def test_event_conv_reduces_to_2d_convolution():
    """Two frames of events: the second frame's outputs are a 3x3 image cross-correlation.

    Frame A puts one event on every pixel at t = 0 with features F_A; frame B
    repeats the pixels at t = d with zero features.  A frame-B event at pixel x'
    sees exactly the frame-A events of its 3x3 block (offset u = x' - x), each
    decayed by exp(-d / tau), so its output is exp(-d/tau) sum_u F_A[x' - u] W_m(u),
    i.e. a zero-padded 3x3 cross-correlation with the centre tap zero.
    """
    H, Wd, C, P = 6, 7, 3, 2
    rng = np.random.default_rng(11)
    yy, xx = np.meshgrid(np.arange(H), np.arange(Wd), indexing="ij")
    px = np.concatenate([xx.ravel(), xx.ravel()]).astype(np.int32)
    py = np.concatenate([yy.ravel(), yy.ravel()]).astype(np.int32)
    d, tau = 300, 1000.0
    t = np.concatenate([np.zeros(H * Wd), np.full(H * Wd, d)]).astype(np.int32)
    FA = rng.standard_normal((H * Wd, C))
    F = np.concatenate([FA, np.zeros_like(FA)])
    W = rng.standard_normal((8, C, P))
    rp, ci = oracle.events_csr(px, py, t, 1000, 1, Wd, H)
    v = event_basis(px, py, t, rp, ci, tau)
    Y = oracle.conv.forward(rp, ci, v, F, W)[H * Wd:]
    # torch conv2d is a cross-correlation: out[y, x] = sum_{a,b} in[y + a - 1, x + b - 1] k[a, b]
    # input pixel x' - u, so tap (a, b) = (1 - uy, 1 - ux) carries W_m(u)
    k = np.zeros((P, C, 3, 3))
    for uy in (-1, 0, 1):
        for ux in (-1, 0, 1):
            m = int(event_offset_index(ux, uy))
            if m >= 0:
                k[:, :, 1 - uy, 1 - ux] = W[m].T
    img = torch.tensor(FA.reshape(H, Wd, C).transpose(2, 0, 1)[None])
    ref = torch.nn.functional.conv2d(img, torch.tensor(k), padding=1)[0].numpy()
    ref = np.exp(-d / tau) * ref.transpose(1, 2, 0).reshape(H * Wd, P)
    np.testing.assert_allclose(Y, ref, rtol=1e-12, atol=1e-12)


def test_event_conv_equals_deployment_recursion():
    """The training form equals the per-pixel exponential moving average form.

    Section 3.2 gives a second implementation: every pixel keeps a decayed sum
    z of the features of its events and the time of its last update; an output
    event decays the 3x3 block's sums to its own time and applies W_m(u).  With
    a window longer than the stream both forms sum over all earlier events of the
    block.  An output is read before the event's own update (j < i).
    """
    w = workloads.small_events(seed=6, n=700, width=6, height=5, duration_us=4000,
                               window_us=10 ** 6, c=3)
    rp, ci, v = _events_problem(w)
    F, W = w["F"].astype(np.float64), w["W"].astype(np.float64)
    Y = oracle.conv.forward(rp, ci, v, F, W)
    Y_ema, _, _ = oracle.conv.deployment_stream(w["px"], w["py"], w["t"], F, W, w["width"],
                                                w["height"], w["tau"])
    np.testing.assert_allclose(Y, Y_ema, rtol=1e-11, atol=1e-11)


def test_deployment_stream_in_pieces():
    """Feeding the stream in pieces, carrying (z, last), gives the outputs and
    final state of one pass; a lone event reads a zero state; the state of a
    pixel with events at t1 < t2 only is f2 + exp(-(t2 - t1)/tau) f1."""
    w = workloads.small_events(seed=7, n=900, width=7, height=6, duration_us=5000, c=4)
    F, W = w["F"].astype(np.float64), w["W"].astype(np.float64)
    args = (w["width"], w["height"], w["tau"])
    Y, z, last = oracle.conv.deployment_stream(w["px"], w["py"], w["t"], F, W, *args)
    Ys, zs, ls = [], None, None
    for a, b in [(0, 1), (1, 300), (300, 301), (301, 900)]:
        Yp, zs, ls = oracle.conv.deployment_stream(w["px"][a:b], w["py"][a:b], w["t"][a:b],
                                                   F[a:b], W, *args, z=zs, last=ls)
        Ys.append(Yp)
    np.testing.assert_allclose(np.concatenate(Ys), Y, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(zs, z, rtol=1e-13, atol=1e-13)
    assert np.array_equal(ls, last)
    assert np.all(Y[0] == 0)
    px, py, t = np.array([3, 3]), np.array([2, 2]), np.array([100, 250])
    f = np.array([[1.0, 2.0], [0.5, -1.0]])
    _, z2, l2 = oracle.conv.deployment_stream(px, py, t, f, np.zeros((8, 2, 1)), 5, 4, 100.0)
    np.testing.assert_allclose(z2[2, 3], f[1] + np.exp(-1.5) * f[0], rtol=1e-15)
    assert l2[2, 3] == 250 and np.count_nonzero(l2) == 1


# ---------------------------------------------------------------- featureless convolution
def _featureless_case(seed=0, basis=workloads.BASIS_WMONO10):
    w = workloads.small_points(seed=seed, basis=basis)
    rp, ci = oracle.points_csr(w["x_in"], w["in_splits"], w["x_out"], w["out_splits"],
                               w["radius"], w["k_cap"])
    v = oracle.basis.point_values(w["basis"], w["x_in"], w["x_out"], rp, ci, w["radius"], w["M"])
    rng = np.random.default_rng(seed)
    Phi = rng.standard_normal((w["M"], 6))
    return w, rp, ci, v, Phi, rng


@pytest.mark.parametrize("basis", [workloads.BASIS_WMONO10, workloads.BASIS_MONO8])
def test_featureless_is_the_convolution_of_ones(basis):
    """Eq. 9-10 is the general convolution with F = 1 (one input channel of ones)
    and W_m = the m-th row of Phi_0."""
    w, rp, ci, v, Phi, _ = _featureless_case(1, basis)
    Z, _ = oracle.conv.featureless_forward(rp, ci, v, Phi)
    ones = np.ones((w["n_in"], 1))
    Y = oracle.conv.forward(rp, ci, v, ones, Phi[:, None, :])
    assert np.allclose(Z, Y, rtol=1e-12, atol=1e-12)
    dZ = np.random.default_rng(5).standard_normal(Z.shape)
    dPhi = oracle.conv.featureless_backward(rp, ci, v, dZ)
    _, dW = oracle.conv.backward(rp, ci, v, ones, Phi[:, None, :], dZ, w["n_in"])
    assert np.allclose(dPhi, dW[:, 0, :], rtol=1e-12, atol=1e-12)


def test_featureless_hand_case():
    """The weighted hand row (fixture): G~ is the column sums of its values, so
    the constant function sums to 1 and Z = G~ Phi_0 by hand."""
    with open(os.path.join(os.path.dirname(__file__), "golden",
                           "points_weighted_hand_case.json")) as f:
        g = json.load(f)
    from fractions import Fraction
    v = np.array([[float(Fraction(x)) for x in row] for row in g["v"]])
    Phi = np.zeros((10, 2))
    Phi[0, 0] = 1.0       # Z[:, 0] = G~[:, 0] = 1
    Phi[1, 1] = 17.0      # Z[:, 1] = 17 * G~[:, 1] = 17 * (-2/17 - 5/136) = -21/8
    Z, Gt = oracle.conv.featureless_forward(g["row_ptr"], g["col_idx"], v, Phi)
    assert np.isclose(Z[0, 0], 1.0, rtol=0, atol=1e-15)
    assert np.isclose(Z[0, 1], -21.0 / 8.0, rtol=0, atol=1e-14)


def test_featureless_adjoint_and_linearity():
    w, rp, ci, v, Phi, rng = _featureless_case(2)
    Z, _ = oracle.conv.featureless_forward(rp, ci, v, Phi)
    dZ = rng.standard_normal(Z.shape)
    dPhi = oracle.conv.featureless_backward(rp, ci, v, dZ)
    assert np.isclose((Z * dZ).sum(), (Phi * dPhi).sum(), rtol=1e-12)
    Z2, _ = oracle.conv.featureless_forward(rp, ci, v, 2.0 * Phi - 1.0)
    Z1, _ = oracle.conv.featureless_forward(rp, ci, v, np.ones_like(Phi))
    assert np.allclose(Z2, 2.0 * Z - Z1, rtol=1e-12, atol=1e-12)
