"""Pins of the oracle's event neighbourhoods and event basis (CPU only)."""
import json
import os

import numpy as np
import pytest

import oracle
import workloads

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _gold():
    with open(os.path.join(GOLD, "events_hand_case.json")) as f:
        return json.load(f)


@pytest.mark.parametrize("method", ["pixels", "scan", "quadratic"])
def test_hand_case_csr(method):
    g = _gold()
    rp, ci = oracle.events_csr(g["px"], g["py"], g["t"], g["window"], 1, 10, 10, method=method)
    assert rp.tolist() == g["row_ptr"] and ci.tolist() == g["col_idx"]


def test_hand_case_basis():
    g = _gold()
    v = oracle.basis.event_basis(g["px"], g["py"], g["t"], np.array(g["row_ptr"]),
                                 np.array(g["col_idx"]), g["tau"])
    for e, (m, ex) in enumerate(zip(g["edge_basis_index"], g["edge_decay_exponent"])):
        want = np.zeros(8)
        if m >= 0:
            want[m] = np.exp(ex)
        assert np.array_equal(v[e], want)


def test_offset_index_table():
    g = _gold()
    for key, m in g["offset_to_index"].items():
        ux, uy = (int(s) for s in key.split(","))
        assert int(oracle.basis.event_offset_index(ux, uy)) == m


def _stream(seed, n, width, height, duration, ties=False):
    rng = np.random.default_rng(seed)
    t = np.sort(rng.integers(0, duration, size=n))
    if ties:                      # many equal timestamps
        t = (t // 50) * 50
    return (rng.integers(0, width, size=n).astype(np.int32),
            rng.integers(0, height, size=n).astype(np.int32), t.astype(np.int32))


@pytest.mark.parametrize("seed,ties,h", [(0, False, 1), (1, True, 1), (2, True, 2), (3, False, 0)])
def test_three_enumerations_agree(seed, ties, h):
    """Per-pixel lists == windowed scan == every earlier event tested."""
    px, py, t = _stream(seed, 3000, 9, 7, 6000, ties)   # small sensor: border pixels everywhere
    ref = oracle.events_csr(px, py, t, 700, h, method="quadratic")
    for m in ("scan", "pixels"):
        got = oracle.events_csr(px, py, t, 700, h, 9, 7, method=m)
        assert np.array_equal(ref[0], got[0]) and np.array_equal(ref[1], got[1])


def test_window_is_inclusive_and_backwards_only():
    px = np.array([3, 3, 3, 3], np.int32)
    py = np.array([3, 3, 4, 3], np.int32)
    t = np.array([0, 100, 100, 200], np.int32)
    rp, ci = oracle.events_csr(px, py, t, 100, 1, 8, 8)
    # e1: e0 at dt = 100 (inclusive); e2: e1 (same time, earlier in order), e0 at dt 100;
    # e3: e1, e2 at dt 100; e0 at dt 200 is out
    assert rp.tolist() == [0, 0, 1, 3, 5] and ci.tolist() == [0, 0, 1, 1, 2]


def test_time_and_space_translation_invariance():
    px, py, t = _stream(4, 2000, 12, 10, 5000, ties=True)
    a = oracle.events_csr(px, py, t, 400, 1, 12, 10)
    b = oracle.events_csr(px, py, t + 12345, 400, 1, 12, 10)
    c = oracle.events_csr(px + 3, py + 2, t, 400, 1, 15, 12)
    for other in (b, c):
        assert np.array_equal(a[0], other[0]) and np.array_equal(a[1], other[1])


def test_unsorted_time_rejected():
    with pytest.raises(ValueError):
        oracle.events_csr(np.zeros(3, np.int32), np.zeros(3, np.int32),
                          np.array([0, 5, 4], np.int32), 10)


def test_event_basis_closed_forms():
    w = workloads.small_events(seed=1)
    rp, ci = oracle.events_csr(w["px"], w["py"], w["t"], w["window"], 1, w["width"], w["height"])
    v = oracle.basis.event_basis(w["px"], w["py"], w["t"], rp, ci, w["tau"])
    rows = oracle.basis.edge_rows(rp)
    same_pixel = (w["px"][rows] == w["px"][ci]) & (w["py"][rows] == w["py"][ci])
    dt = (w["t"][rows] - w["t"][ci]).astype(np.float64)
    assert np.all(v[same_pixel] == 0)
    nz = np.count_nonzero(v, axis=1)
    assert np.all(nz[~same_pixel] == 1)
    np.testing.assert_allclose(v.sum(axis=1)[~same_pixel], np.exp(-dt[~same_pixel] / w["tau"]),
                               rtol=1e-15, atol=0)


# ---------------------------------------------------------------- learned decays (Eq. 12, M_v > 1)
def _decay_problem(seed=0, n=900, Mv=2):
    w = workloads.small_events(seed=seed, n=n, width=7, height=6, duration_us=6000,
                               window_us=2500, c=3)
    rp, ci = oracle.events_csr(w["px"], w["py"], w["t"], w["window"], 1, w["width"], w["height"])
    rng = np.random.default_rng(seed)
    lam = rng.uniform(0.2, 3.0, size=(8, Mv)) / w["tau"]
    return w, rp, ci, lam


def test_single_decay_is_the_fixed_event_basis():
    """M_v = 1 with lambda = 1/tau everywhere is the fixed-decay basis exactly."""
    w, rp, ci, _ = _decay_problem(1)
    lam = np.full((8, 1), 1.0 / w["tau"])
    v = oracle.basis.event_decay_basis(w["px"], w["py"], w["t"], rp, ci, lam)
    v0 = oracle.basis.event_basis(w["px"], w["py"], w["t"], rp, ci, w["tau"])
    assert np.allclose(v, v0, rtol=1e-14, atol=0)


def test_decays_equal_the_deployment_recursion():
    """Eq. 13-15 with M_v = 2 decays per offset: every pixel keeps one decayed
    sum per (offset, decay); an output decays the block's sums to its own time
    and applies Theta_uv.  With a window longer than the stream both forms sum
    over all earlier events of the block."""
    w = workloads.small_events(seed=7, n=500, width=5, height=4, duration_us=3000,
                               window_us=10 ** 6, c=3)
    rp, ci = oracle.events_csr(w["px"], w["py"], w["t"], w["window"], 1, w["width"], w["height"])
    rng = np.random.default_rng(3)
    Mv = 2
    lam = rng.uniform(0.5, 4.0, size=(8, Mv)) / 1000.0
    v = oracle.basis.event_decay_basis(w["px"], w["py"], w["t"], rp, ci, lam)
    F = w["F"].astype(np.float64)
    W = rng.standard_normal((8 * Mv, w["C_in"], 2))
    Y = oracle.conv.forward(rp, ci, v, F, W)
    Y_ema, z, _ = oracle.conv.deployment_stream(w["px"], w["py"], w["t"], F, W, w["width"],
                                                w["height"], None, decays=lam)
    np.testing.assert_allclose(Y, Y_ema, rtol=1e-11, atol=1e-11)
    assert z.shape == (w["height"], w["width"], 8, Mv, w["C_in"])


def test_equal_decays_deploy_as_the_fixed_form():
    """With every lambda_uv = 1/tau the per-(offset, decay) states of a pixel
    coincide, and the learned-decay deployment form equals the fixed-decay one
    with W_u = sum_v W_(u,v); fed in pieces it carries its state like one pass."""
    w = workloads.small_events(seed=8, n=600, width=6, height=5, duration_us=4000, c=3)
    rng = np.random.default_rng(9)
    Mv = 3
    lam = np.full((8, Mv), 1.0 / w["tau"])
    F = w["F"].astype(np.float64)
    W = rng.standard_normal((8 * Mv, w["C_in"], 4))
    args = (w["width"], w["height"], w["tau"])
    Y, z, last = oracle.conv.deployment_stream(w["px"], w["py"], w["t"], F, W, *args, decays=lam)
    Y0, z0, last0 = oracle.conv.deployment_stream(w["px"], w["py"], w["t"], F,
                                                  W.reshape(8, Mv, w["C_in"], 4).sum(axis=1),
                                                  *args)
    np.testing.assert_allclose(Y, Y0, rtol=1e-11, atol=1e-11)
    for u in range(8):
        for v in range(Mv):
            np.testing.assert_allclose(z[:, :, u, v], z0, rtol=1e-13, atol=1e-13)
    assert np.array_equal(last, last0)
    lam2 = rng.uniform(0.5, 3.0, size=(8, Mv)) / w["tau"]
    Y2, z2, l2 = oracle.conv.deployment_stream(w["px"], w["py"], w["t"], F, W, *args, decays=lam2)
    Ys, zs, ls = [], None, None
    for a, b in [(0, 250), (250, 251), (251, 600)]:
        Yp, zs, ls = oracle.conv.deployment_stream(w["px"][a:b], w["py"][a:b], w["t"][a:b], F[a:b],
                                                   W, *args, z=zs, last=ls, decays=lam2)
        Ys.append(Yp)
    np.testing.assert_allclose(np.concatenate(Ys), Y2, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(zs, z2, rtol=1e-13, atol=1e-13)


def test_decay_gradient_matches_finite_differences():
    w, rp, ci, lam = _decay_problem(2, Mv=2)
    F = w["F"].astype(np.float64)
    rng = np.random.default_rng(4)
    W = rng.standard_normal((16, w["C_in"], 4))
    dY = rng.standard_normal((w["n_out"], 4))

    def loss(l):
        v = oracle.basis.event_decay_basis(w["px"], w["py"], w["t"], rp, ci, l)
        return float((oracle.conv.forward(rp, ci, v, F, W) * dY).sum())

    vd = oracle.basis.event_decay_basis(w["px"], w["py"], w["t"], rp, ci, lam, derivative=True)
    g = oracle.conv.decay_backward(rp, ci, vd, F, W, dY)
    for m in [0, 5, 11, 15]:
        u, q = divmod(m, 2)
        h = 1e-4 * lam[u, q]
        lp, lm = lam.copy(), lam.copy()
        lp[u, q] += h
        lm[u, q] -= h
        fd = (loss(lp) - loss(lm)) / (2 * h)
        assert np.isclose(g[m], fd, rtol=1e-6, atol=1e-9 * max(1.0, abs(fd)))


def _brute_block_pattern(px, py, t, window, h, reverse):
    """Rows (reverse: columns) from the definition, each in block order: the
    (2h+1)^2 pixels around the centre event row-major, then stream order."""
    n = len(t)
    out = []
    for c in range(n):
        ent = []
        for o in range(n):
            later, earlier = (o, c) if reverse else (c, o)
            if not (earlier < later and 0 <= int(t[later]) - int(t[earlier]) <= window):
                continue
            dx, dy = int(px[o]) - int(px[c]), int(py[o]) - int(py[c])
            if abs(dx) <= h and abs(dy) <= h:
                ent.append(((dy + h) * (2 * h + 1) + (dx + h), o))
        out.append([o for _, o in sorted(ent)])
    return out


@pytest.mark.parametrize("h", [1, 2])
def test_rows_and_columns_in_block_order(h):
    """Rows and columns of the event pattern against a brute force written from
    the definition: a row holds the earlier events of its block within the
    window, a column the later ones, each listed pixel by pixel (row-major
    around the centre event) and in stream order within a pixel."""
    rng = np.random.default_rng(60 + h)
    n, W, H = 400, 6, 5
    px = rng.integers(0, W, n).astype(np.int32)
    py = rng.integers(0, H, n).astype(np.int32)
    t = np.sort(rng.integers(0, 5000, n)).astype(np.int32)
    rp, ci = oracle.events_csr(px, py, t, 300, h, W, H)
    cp, ri = oracle.events_csc(px, py, t, 300, h, W, H)
    rows = _brute_block_pattern(px, py, t, 300, h, False)
    cols = _brute_block_pattern(px, py, t, 300, h, True)
    assert [ci[rp[i]:rp[i + 1]].tolist() for i in range(n)] == rows
    assert [ri[cp[j]:cp[j + 1]].tolist() for j in range(n)] == cols
    assert any(r != sorted(r) for r in rows)      # the order is not the index order


def test_block_order_hand_case():
    """Event 3 at (2, 2) sees event 0 at (3, 2) (position 5 of its 3x3 block),
    event 1 at (1, 1) (position 0) and event 2 at (2, 2) (position 4, its own
    pixel): its row is [1, 2, 0].  Event 0's column holds events 2 and 3, both
    at position 3 around it, in stream order.  In the second stream event 0 at
    (2, 2) is seen by event 1 at (3, 3) (position 8 around event 0) and event 2
    at (1, 1) (position 0): its column is [2, 1]."""
    px = np.array([3, 1, 2, 2], np.int32)
    py = np.array([2, 1, 2, 2], np.int32)
    t = np.array([0, 1, 2, 3], np.int32)
    rp, ci = oracle.events_csr(px, py, t, 100, 1, 5, 5)
    assert ci[rp[3]:rp[4]].tolist() == [1, 2, 0]
    cp, ri = oracle.events_csc(px, py, t, 100, 1, 5, 5)
    assert ri[cp[0]:cp[1]].tolist() == [2, 3]
    px = np.array([2, 3, 1], np.int32)
    py = np.array([2, 3, 1], np.int32)
    cp, ri = oracle.events_csc(px, py, np.array([0, 1, 2], np.int32), 100, 1, 5, 5)
    assert ri[cp[0]:cp[1]].tolist() == [2, 1]
