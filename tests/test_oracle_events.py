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
