"""Pins of the oracle's subsampling (CPU only): farthest points against a
brute-force recomputation, rejection sampling against the characterisation of
the lexicographically first maximal independent set it computes, and the
neighbourhood-limited variant against the exact one when the neighbourhood
covers the cloud."""
import numpy as np
import pytest

import oracle
import workloads


def _d2(a, b):
    d = np.asarray(a, np.float32) - np.asarray(b, np.float32)
    return (d[..., 0] * d[..., 0] + d[..., 1] * d[..., 1]) + d[..., 2] * d[..., 2]


def _clouds(seed, sizes, scale=1.0):
    rng = np.random.default_rng(seed)
    xs = [workloads.ellipsoid_surface_points(rng, n, rng.uniform(0.5, 1.0, size=3)) * scale
          if n else np.zeros((0, 3)) for n in sizes]
    x = np.concatenate(xs).astype(np.float32)
    splits = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    return x, splits


@pytest.mark.parametrize("seed", [0, 1])
def test_ifp_matches_brute_force(seed):
    x, splits = _clouds(seed, [37, 1, 25])
    counts = [12, 1, 25]
    got, _ = oracle.sampling.ifp(x, splits, counts)
    k = 0
    for b in range(3):
        s, e = splits[b], splits[b + 1]
        chosen = []
        for _ in range(counts[b]):
            # the distance of every point to its nearest chosen point, afresh
            best, arg = -1.0, -1
            for j in range(s, e):
                dj = min((_d2(x[j], x[c]) for c in chosen), default=np.float32(np.inf))
                if dj > best:
                    best, arg = dj, j
            chosen.append(arg)
        assert got[k:k + counts[b]].tolist() == chosen
        assert chosen[0] == s                  # all distances infinite: the first point
        k += counts[b]


def _ball(x, splits, radius):
    return oracle.points_csr(x, splits, x, splits, radius, 0)


@pytest.mark.parametrize("seed,radius", [(0, 0.3), (1, 0.15)])
def test_rejection_sampling_is_the_first_maximal_independent_set(seed, radius):
    x, splits = _clouds(seed, [300, 0, 450])
    rp, ci = _ball(x, splits, radius)
    taken, dmin = oracle.sampling.rejection_sampling(x, splits, rp, ci)
    for i in range(len(x)):
        nb = ci[rp[i]:rp[i + 1]]
        earlier_taken = [k for k in nb if k < i and taken[k]]
        if taken[i]:
            assert not earlier_taken               # independent, first in scan order
        else:
            assert earlier_taken                   # dominated by an earlier sample
        # d_min: the nearest taken neighbour (itself, at 0, when taken)
        want = min(_d2(x[i], x[k]) for k in nb if taken[k])
        assert dmin[i] == want
    assert taken.sum() < len(x)


def test_approx_ifp_with_a_covering_neighbourhood_is_exact_ifp():
    x, splits = _clouds(2, [120, 80])
    rp, ci = _ball(x, splits, 10.0)            # every point neighbours every other
    counts = [30, 17]
    a_idx, a_d = oracle.sampling.approx_ifp(x, splits, counts, rp, ci)
    e_idx, e_d = oracle.sampling.ifp(x, splits, counts)
    assert np.array_equal(a_idx, e_idx) and np.array_equal(a_d, e_d)


def test_approx_ifp_after_rejection_takes_the_farthest_first():
    x, splits = _clouds(3, [400])
    rp, ci = _ball(x, splits, 0.2)
    taken, dmin = oracle.sampling.rejection_sampling(x, splits, rp, ci)
    extra, _ = oracle.sampling.approx_ifp(x, splits, [5], rp, ci, dmin)
    assert not taken[extra[0]]
    assert dmin[extra[0]] == dmin.max()
    assert int(np.argmax(dmin)) == extra[0]


def test_approx_ifp_after_rejection_concatenates():
    x, splits = _clouds(4, [500, 30])
    rp, ci = _ball(x, splits, 0.2)
    taken, dmin = oracle.sampling.rejection_sampling(x, splits, rp, ci)
    idx, _ = oracle.sampling.approx_ifp_after_rejection(x, splits, 200, rp, ci)
    n0 = int(taken[:500].sum())
    assert n0 < 200
    assert idx[:n0].tolist() == np.nonzero(taken[:500])[0].tolist()
    assert len(set(idx[:200].tolist())) == 200          # the extra points are new
    # the small cloud keeps only its first 30 points' worth (all of it)
    assert sorted(idx[200:].tolist()) == list(range(500, 530))
