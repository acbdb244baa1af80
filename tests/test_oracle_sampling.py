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


def _farthest_remaining(x, s, e, count):
    """Brute force: each step recomputes every remaining point's distance to
    its nearest chosen point and takes the largest (lowest index on ties)."""
    chosen = []
    for _ in range(count):
        best, arg = -1.0, -1
        for j in range(s, e):
            if j in chosen:
                continue
            dj = min((_d2(x[j], x[c]) for c in chosen), default=np.float32(np.inf))
            if dj > best:
                best, arg = dj, j
        chosen.append(arg)
    return chosen


@pytest.mark.parametrize("seed", [0, 1])
def test_ifp_matches_brute_force(seed):
    x, splits = _clouds(seed, [37, 1, 25])
    counts = [12, 1, 25]
    got, _ = oracle.sampling.ifp(x, splits, counts)
    k = 0
    for b in range(3):
        s, e = splits[b], splits[b + 1]
        chosen = _farthest_remaining(x, s, e, counts[b])
        assert got[k:k + counts[b]].tolist() == chosen
        assert chosen[0] == s                  # all distances infinite: the first point
        k += counts[b]


def _doubled(seed, n):
    """A cloud of n distinct points followed by a copy of each."""
    x, _ = _clouds(seed, [n])
    return np.concatenate([x, x]), np.array([0, 2 * n], np.int32)


def test_coincident_points_are_each_taken_once():
    """With every point doubled, asking for the whole cloud takes every index
    once: after the distinct points the remaining distances are all 0, and
    the farthest remaining point is the lowest remaining index.  Exact IFP
    against the brute force; the ball-limited variant and rejection followed
    by it give permutations."""
    x, splits = _doubled(5, 20)
    got, d = oracle.sampling.ifp(x, splits, [40])
    assert got.tolist() == _farthest_remaining(x, 0, 40, 40)
    assert sorted(got.tolist()) == list(range(40)) and not d.any()
    assert sorted(got[20:].tolist()) == list(range(20, 40))    # the copies come last
    rp, ci = _ball(x, splits, 0.3)
    a, _ = oracle.sampling.approx_ifp(x, splits, [40], rp, ci)
    assert sorted(a.tolist()) == list(range(40))
    r, _ = oracle.sampling.approx_ifp_after_rejection(x, splits, 40, rp, ci)
    assert sorted(r.tolist()) == list(range(40))


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



# ---------------------------------------------------------------- LIF event sampler
def _lif(px, py, t, W, H, k, S, decay, th, rs):
    return oracle.sampling.lif(np.asarray(px, np.int32), np.asarray(py, np.int32),
                               np.asarray(t, np.int32), W, H, k, S, decay, th, rs)


def test_lif_without_decay_fires_every_third_event():
    """One pixel, one cell (kernel 1, stride 1), no decay: the potential climbs
    by 1 per event, so with threshold 2.5 and reset 0 every third event fires."""
    out = _lif([0] * 10, [0] * 10, range(10), 1, 1, 1, 1, np.inf, 2.5, 0.0)
    assert out[:, 0].tolist() == [2, 5, 8]
    assert (out[:, 1:] == 0).all()


def test_lif_decay_threshold_closed_form():
    """Two events at one pixel, gap g: the second fires iff exp(-g / decay) + 1
    exceeds the threshold, i.e. g < decay * ln(1 / (thresh - 1))."""
    decay, thresh = 100.0, 1.5
    g0 = decay * np.log(1.0 / (thresh - 1.0))      # 69.3...
    for g, fires in [(60, True), (69, True), (70, False), (200, False)]:
        out = _lif([0, 0], [0, 0], [0, g], 1, 1, 1, 1, decay, thresh, 0.0)
        assert (len(out) == 1) == fires and (g < g0) == fires


def test_lif_first_spike_of_a_regular_train():
    """Events every D at one neuron with no reset before the first spike: after
    m events the potential is the geometric sum (1 - a^m) / (1 - a), a =
    exp(-D / decay), so the first spike is at the first m where that sum
    exceeds the threshold."""
    D, decay = 30, 100.0
    a = np.exp(-D / decay)
    for thresh in [1.2, 2.0, 3.1, 3.8]:
        m = next(m for m in range(1, 200) if (1 - a ** m) / (1 - a) > thresh)
        out = _lif([0] * 60, [0] * 60, np.arange(60) * D, 1, 1, 1, 1, decay, thresh, -5.0)
        assert out[0, 0] == m - 1


def test_lif_overlapping_fields_share_the_event():
    """Kernel 3, stride 2 on a 6 x 6 sensor (3 x 3 cells, cell o seeing inputs
    2o-1 .. 2o+1): input (3, 3) reaches cells 1 and 2 in each dimension, so each
    of the four gains 1/4 per event and, with threshold 1, they fire together
    at the fifth event, listed row-major.  Input (2, 2) reaches cell (1, 1)
    alone and fires at its second event."""
    out = _lif([3] * 5, [3] * 5, [0] * 5, 6, 6, 3, 2, 1e9, 1.0, 0.0)
    # potentials 0.25, 0.5, 0.75, 1.0 (not above 1), 1.25 -> fire at event 4
    assert out.tolist() == [[4, 1, 1], [4, 2, 1], [4, 1, 2], [4, 2, 2]]
    out = _lif([2] * 3, [2] * 3, [0] * 3, 6, 6, 3, 2, 1e9, 1.0, 0.0)
    assert out.tolist() == [[1, 1, 1]]


def test_lif_border_and_unreached_inputs():
    """On the border an input reaches fewer cells (n is smaller, so each gains
    more); with a stride above the kernel some inputs reach no cell at all and
    change nothing."""
    # x = 5 on a 6-wide sensor: cell 2 (3 .. 5) only, cell 3 is off the grid
    out = _lif([5] * 2, [0] * 2, [0] * 2, 6, 1, 3, 2, np.inf, 1.5, 0.0)
    assert out.tolist() == [[1, 2, 0]]
    # kernel 1, stride 2: odd inputs are seen by no cell
    out = _lif([1, 1, 1, 0, 0], [0] * 5, range(5), 4, 1, 1, 2, np.inf, 1.5, 0.0)
    assert out.tolist() == [[4, 0, 0]]


def test_lif_cells_are_independent():
    """Each output cell's spikes depend only on the events of its receptive
    field: simulating one cell at a time over its own events, with the cell
    windows and n counted by brute force here, gives the same output events,
    in the order (input event, oy, ox)."""
    rng = np.random.default_rng(9)
    n, W, H = 3000, 12, 9
    px = rng.integers(0, W, n)
    py = rng.integers(0, H, n)
    t = np.sort(rng.integers(0, 20000, n))
    k, S, decay, th, rs = 3, 2, 800.0, 0.9, 0.1
    full = _lif(px, py, t, W, H, k, S, decay, th, rs)
    Wo, Ho = -(-W // S), -(-H // S)
    inside = lambda x, o: o * S - 1 <= x <= o * S + 1
    got = []
    for oy in range(Ho):
        for ox in range(Wo):
            V = Tm = 0.0
            for i in range(n):
                if not (inside(px[i], ox) and inside(py[i], oy)):
                    continue
                nn = (sum(inside(px[i], o) for o in range(Wo)) *
                      sum(inside(py[i], o) for o in range(Ho)))
                v = V * np.exp(-(float(t[i]) - Tm) / decay) + 1.0 / nn
                if v > th:
                    v = rs
                    got.append((i, ox, oy))
                V, Tm = v, float(t[i])
    got.sort(key=lambda r: (r[0], r[2], r[1]))
    assert len(got) > 100
    assert [tuple(r) for r in full.tolist()] == got
