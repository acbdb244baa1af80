"""Pins of the oracle's point neighbourhoods and point basis (CPU only).

Each test checks the oracle against something other than itself: a
hand-computed case, a KD-tree library search, or an invariant that the ball
neighbourhood of Section 3.1 must satisfy.
"""
import json
import os

import numpy as np
import pytest
from scipy.spatial import cKDTree

import oracle
import workloads

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def _single(x_in, x_out):
    return (np.asarray(x_in, np.float32), np.array([0, len(x_in)], np.int32),
            np.asarray(x_out, np.float32), np.array([0, len(x_out)], np.int32))


def test_hand_case_csr():
    g = _gold("points_hand_case.json")
    x_in, s_in, x_out, s_out = _single(g["x_in"], g["x_out"])
    rp, ci = oracle.points_csr(x_in, s_in, x_out, s_out, g["radius"], 0)
    assert rp.tolist() == g["uncapped"]["row_ptr"]
    assert ci.tolist() == g["uncapped"]["col_idx"]
    rp2, ci2 = oracle.points_csr(x_in, s_in, x_out, s_out, g["radius"], g["cap2"]["k_cap"])
    assert rp2.tolist() == g["cap2"]["row_ptr"]
    assert ci2.tolist() == g["cap2"]["col_idx"]


def test_hand_case_basis_exact():
    g = _gold("points_hand_case.json")
    rp = np.array(g["uncapped"]["row_ptr"], np.int32)
    ci = np.array(g["uncapped"]["col_idx"], np.int32)
    v = oracle.basis.point_basis(np.array(g["x_in"], np.float32), np.array(g["x_out"], np.float32),
                                 rp, ci, g["radius"], 4)
    assert v.tolist() == g["uncapped"]["v"]


def _dyadic_cloud(rng, n, scale=1.0, bits=12):
    """Coordinates on a 2^-bits grid, so float32 differences and squares are exact."""
    lim = int(scale * (1 << bits))
    q = rng.integers(-lim, lim + 1, size=(n, 3))
    return (q / float(1 << bits)).astype(np.float32)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_uncapped_ball_matches_kdtree(seed):
    """The uncapped ball equals scipy's KD-tree ball query (the paper's CPU search)."""
    rng = np.random.default_rng(seed)
    x = _dyadic_cloud(rng, 700, scale=0.6)
    y = _dyadic_cloud(rng, 180, scale=0.6)
    r = 0.1875                      # dyadic: r*r is exact in float32
    rp, ci = oracle.points_csr(x, np.array([0, 700], np.int32), y,
                               np.array([0, 180], np.int32), r, 0)
    tree = cKDTree(x.astype(np.float64))
    # exact squared distances are multiples of 2^-24; the largest one below r^2
    # is r^2 - 2^-24, so a query radius between the two is a strict test
    rq = np.sqrt(r * r - 2.0 ** -25)
    for i in range(len(y)):
        want = sorted(tree.query_ball_point(y[i].astype(np.float64), rq))
        assert list(ci[rp[i]:rp[i + 1]]) == want


def test_points_on_the_sphere_exactly_at_radius_are_excluded():
    x_out = np.zeros((1, 3), np.float32)
    x_in = np.array([[0.25, 0, 0], [0, -0.25, 0], [0, 0, 0.25], [0.2490234375, 0, 0]], np.float32)
    rp, ci = oracle.points_csr(x_in, np.array([0, 4], np.int32), x_out,
                               np.array([0, 1], np.int32), 0.25, 0)
    assert ci.tolist() == [3]


@pytest.mark.parametrize("k_cap", [1, 3, 7])
def test_cap_keeps_the_k_smallest(k_cap):
    """Capped rows are the k smallest (d2, j) of the uncapped rows, sorted by j."""
    rng = np.random.default_rng(10 + k_cap)
    x = _dyadic_cloud(rng, 400, scale=0.5, bits=6)   # coarse grid: many distance ties
    splits = np.array([0, 400], np.int32)
    r = 0.25
    rp_u, ci_u = oracle.points_csr(x, splits, x, splits, r, 0)
    rp_c, ci_c = oracle.points_csr(x, splits, x, splits, r, k_cap)
    xd = x.astype(np.float64)
    for i in range(len(x)):
        full = ci_u[rp_u[i]:rp_u[i + 1]]
        kept = ci_c[rp_c[i]:rp_c[i + 1]]
        assert list(kept) == sorted(kept)
        assert len(kept) == min(k_cap, len(full))
        assert set(kept) <= set(full)
        d2 = {j: float(np.sum((xd[i] - xd[j]) ** 2)) for j in full}   # exact on this grid
        dropped = [j for j in full if j not in set(kept)]
        if kept.size and dropped:
            worst_kept = max((d2[j], j) for j in kept)
            best_dropped = min((d2[j], j) for j in dropped)
            assert worst_kept < best_dropped


def test_translation_invariance_bitwise():
    rng = np.random.default_rng(5)
    x = _dyadic_cloud(rng, 500, scale=0.9)
    splits = np.array([0, 500], np.int32)
    a = oracle.points_csr(x, splits, x[:200], np.array([0, 200], np.int32), 0.15625, 9)
    xs = (x.astype(np.float64) + 0.5).astype(np.float32)
    b = oracle.points_csr(xs, splits, xs[:200], np.array([0, 200], np.int32), 0.15625, 9)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_permutation_equivariance():
    rng = np.random.default_rng(6)
    x = _dyadic_cloud(rng, 300, scale=0.7)
    splits = np.array([0, 300], np.int32)
    y = x[:90]
    rp, ci = oracle.points_csr(x, splits, y, np.array([0, 90], np.int32), 0.2, 0)
    perm = rng.permutation(300)
    rp2, ci2 = oracle.points_csr(x[perm], splits, y, np.array([0, 90], np.int32), 0.2, 0)
    assert np.array_equal(rp, rp2)
    for i in range(90):
        assert sorted(perm[ci2[rp2[i]:rp2[i + 1]]]) == list(ci[rp[i]:rp[i + 1]])


def test_ball_symmetry_in_place():
    """In-place uncapped balls are symmetric (Section 3.1, 'Symmetry')."""
    w = workloads.small_points(seed=3, k_cap=0)
    rp, ci = oracle.points_csr(w["x_in"], w["in_splits"], w["x_out"], w["out_splits"],
                               w["radius"], 0)
    cp, ri, perm = oracle.csr_transpose(rp, ci, w["n_in"])
    assert np.array_equal(cp, rp) and np.array_equal(ri, ci)
    # even monomials agree across the transpose, odd ones change sign
    v = oracle.basis.point_basis(w["x_in"], w["x_out"], rp, ci, w["radius"], 8)
    vt = v[perm]
    sign = np.array([1, -1, -1, -1, 1, 1, 1, 1], np.float64)
    np.testing.assert_allclose(vt * sign, v, rtol=0, atol=1e-15)


def test_ragged_batch_is_block_diagonal():
    w = workloads.small_points(seed=4, n_out=40)
    rp, ci = oracle.points_csr(w["x_in"], w["in_splits"], w["x_out"], w["out_splits"],
                               w["radius"], w["k_cap"])
    for b in range(len(w["in_splits"]) - 1):
        i0, i1 = w["in_splits"][b], w["in_splits"][b + 1]
        o0, o1 = w["out_splits"][b], w["out_splits"][b + 1]
        rb, cb = oracle.points_csr(w["x_in"][i0:i1], np.array([0, i1 - i0], np.int32),
                                   w["x_out"][o0:o1], np.array([0, o1 - o0], np.int32),
                                   w["radius"], w["k_cap"])
        seg = ci[rp[o0]:rp[o1]]
        assert np.array_equal(seg - i0, cb)
        assert np.array_equal(rp[o0:o1 + 1] - rp[o0], rb)


def test_empty_clouds_and_rows():
    x = np.array([[0, 0, 0], [0.05, 0, 0]], np.float32)
    far = np.array([[10, 10, 10]], np.float32)
    x_out = np.concatenate([far, x])
    in_splits = np.array([0, 0, 2], np.int32)      # first cloud has no inputs
    out_splits = np.array([0, 1, 3], np.int32)
    rp, ci = oracle.points_csr(x, in_splits, x_out, out_splits, 0.1, 0)
    assert rp.tolist() == [0, 0, 2, 4] and ci.tolist() == [0, 1, 0, 1]
    rp, ci = oracle.points_csr(np.zeros((0, 3), np.float32), np.array([0, 0], np.int32),
                               np.zeros((0, 3), np.float32), np.array([0, 0], np.int32), 0.1, 4)
    assert rp.tolist() == [0] and len(ci) == 0


def test_transpose_matches_stable_sort():
    w = workloads.small_points(seed=7, n_out=50)
    rp, ci = oracle.points_csr(w["x_in"], w["in_splits"], w["x_out"], w["out_splits"],
                               w["radius"], w["k_cap"])
    cp, ri, perm = oracle.csr_transpose(rp, ci, w["n_in"])
    order = np.argsort(ci, kind="stable")
    rows = np.repeat(np.arange(len(rp) - 1), np.diff(rp))
    assert np.array_equal(perm, order)
    assert np.array_equal(ri, rows[order])
    assert np.array_equal(cp, np.concatenate([[0], np.cumsum(np.bincount(ci, minlength=w["n_in"]))]))


def test_basis_closed_forms():
    x_in = np.array([[0, 0, 0], [0.25, 0, 0], [0, 0.125, 0.125]], np.float32)
    x_out = np.zeros((1, 3), np.float32)
    rp = np.array([0, 3], np.int32)
    ci = np.array([0, 1, 2], np.int32)
    v = oracle.basis.point_basis(x_in, x_out, rp, ci, 0.25, 8)
    assert v[0].tolist() == [1, 0, 0, 0, 0, 0, 0, 0]       # zero edge vector
    assert np.all(v[1] == 0)                                  # |u| = 1: window vanishes
    # u = (0, -0.5, -0.5): |u|^2 = 0.5, w = 0.25
    assert v[2].tolist() == [0.25, 0, -0.125, -0.125, 0, 0.0625, 0.0625, 0]


def test_mono8_hand_case_every_column():
    """Each of the eight M = 8 columns at an edge whose components are all
    nonzero with distinct magnitudes (exact fractions in the fixture): the
    eighth column is ux*uy*w, not one of the monomials the set leaves out."""
    from fractions import Fraction
    g = _gold("points_mono8_hand_case.json")
    x_in, s_in, x_out, s_out = _single(g["x_in"], g["x_out"])
    rp, ci = oracle.points_csr(x_in, s_in, x_out, s_out, g["radius"], 0)
    assert rp.tolist() == [0, 1] and ci.tolist() == [0]
    v = oracle.basis.point_basis(x_in, x_out, rp, ci, g["radius"], 8)
    want = [float(Fraction(x)) for x in g["v"]]
    assert v[0].tolist() == want
    for other in g["left_out"].values():
        assert v[0, 7] != float(Fraction(other))
    # the values are pairwise distinct, so a swap of two columns shows
    assert len(set(np.abs(v[0]).tolist())) == 8


# ---------------------------------------------------------------- weighted convolution (Eq. 11)
def _frac(x):
    from fractions import Fraction
    return float(Fraction(x))


def test_weighted_hand_case():
    """Eq. 11 with the M = 10 monomials on a hand-computed row (fractions in the fixture)."""
    g = _gold("points_weighted_hand_case.json")
    x_in, s_in, x_out, s_out = _single(g["x_in"], g["x_out"])
    rp, ci = oracle.points_csr(x_in, s_in, x_out, s_out, g["radius"], 0)
    assert rp.tolist() == g["row_ptr"] and ci.tolist() == g["col_idx"]
    v = oracle.basis.weighted_point_basis(x_in, x_out, rp, ci, g["radius"])
    want = np.array([[_frac(x) for x in row] for row in g["v"]])
    assert v.shape == (3, 10)
    assert np.allclose(v, want, rtol=1e-15, atol=1e-16)


def _weighted_cloud(seed, n=600, n_out=150, radius=0.3):
    rng = np.random.default_rng(seed)
    x = workloads.ellipsoid_surface_points(rng, n, np.array([1.0, 0.7, 0.5])).astype(np.float32)
    y = x[:n_out]
    s_in = np.array([0, n], np.int32)
    s_out = np.array([0, n_out], np.int32)
    rp, ci = oracle.points_csr(x, s_in, y, s_out, radius, 0)
    return x, y, rp, ci, radius


@pytest.mark.parametrize("seed", [0, 1])
def test_weighted_rows_are_a_partition_of_unity(seed):
    """The constant basis function's values of a row sum to 1 (sum_j w_ij / W_i),
    and a row with one neighbour gets weight exactly 1."""
    x, y, rp, ci, r = _weighted_cloud(seed)
    v = oracle.basis.weighted_point_basis(x, y, rp, ci, r)
    lens = np.diff(rp)
    sums = np.add.reduceat(v[:, 0], rp[:-1][lens > 0])
    assert np.allclose(sums, 1.0, rtol=0, atol=1e-13)
    single = np.nonzero(lens == 1)[0]
    assert np.all(v[rp[single], 0] == 1.0)
    # the weights fall to zero towards the sphere: every value is a weighted
    # monomial of |u| < 1, so no column exceeds 1 in magnitude
    assert np.abs(v).max() <= 1.0


def test_weighted_translation_invariance():
    x, y, rp, ci, r = _weighted_cloud(2)
    shift = np.array([0.5, -0.25, 0.125], np.float64)
    v = oracle.basis.weighted_point_basis(x, y, rp, ci, r)
    v2 = oracle.basis.weighted_point_basis(x.astype(np.float64) + shift,
                                           y.astype(np.float64) + shift, rp, ci, r)
    assert np.allclose(v, v2, rtol=0, atol=1e-12)


def test_weighted_mirror_symmetry():
    """Mirroring x flips exactly the monomials odd in ux: ux, ux*uy, ux*uz."""
    x, y, rp, ci, r = _weighted_cloud(3)
    v = oracle.basis.weighted_point_basis(x, y, rp, ci, r)
    m = np.array([-1.0, 1.0, 1.0])
    vm = oracle.basis.weighted_point_basis(x * m, y * m, rp, ci, r)
    sign = np.array([1, -1, 1, 1, 1, 1, 1, -1, -1, 1], np.float64)
    assert np.allclose(vm, v * sign, rtol=0, atol=1e-13)
    my = np.array([1.0, 1.0, -1.0])
    vz = oracle.basis.weighted_point_basis(x * my, y * my, rp, ci, r)
    sign_z = np.array([1, 1, 1, -1, 1, 1, 1, 1, -1, -1], np.float64)
    assert np.allclose(vz, v * sign_z, rtol=0, atol=1e-13)
