"""Helpers of the GPU parity tests: device copies of workloads, error metrics."""
from __future__ import annotations

import numpy as np
import torch

import paper_2012_01170_amd as sbc

DEV = torch.device("cuda:0")

# Tolerances (relative, row-normwise; see row_error): the float32 path and the
# bf16-input path with float32 accumulation.
TOL_F32 = 1e-5
TOL_BF16 = 2e-2


def dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def dev_features(w, name):
    if w["dtype"] == "bf16":
        bits = np.ascontiguousarray(w[name + "_bits"]).view(np.int16)
        return torch.from_numpy(bits).to(DEV).view(torch.bfloat16)
    return dev(w[name])


def geometry(w, t: dict) -> sbc.Geometry:
    if w["kind"] == "points":
        return sbc.Geometry(w["basis"], radius=w["radius"], x_in=t["x_in"], x_out=t["x_out"])
    if w["basis"] == "event_decays":
        return sbc.Geometry("event_decays", px=t["px"], py=t["py"], t=t["t"],
                            decays=dev(w["decays"]))
    return sbc.Geometry("event8", tau=w["tau"], px=t["px"], py=t["py"], t=t["t"])


def to_device(w) -> dict:
    t = {}
    if w["kind"] == "points":
        for k in ("x_in", "x_out", "in_splits", "out_splits"):
            t[k] = dev(w[k])
    else:
        for k in ("px", "py", "t"):
            t[k] = dev(w[k])
    for k in ("F", "W", "dY"):
        t[k] = dev_features(w, k)
    return t


def search(w, t, sync=True) -> sbc.CSR:
    if w["kind"] == "points":
        return sbc.neighbour_search_points(t["x_in"], t["in_splits"], t["x_out"], t["out_splits"],
                                           w["radius"], w["k_cap"], sync=sync)
    return sbc.neighbour_search_events(t["px"], t["py"], t["t"], w["width"], w["height"],
                                       w["window"], w.get("half_extent", 1), sync=sync)


def row_error(got: np.ndarray, ref: np.ndarray) -> float:
    """max over rows of max|got - ref| / max|ref|; rows with ref == 0 must be exactly 0."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    scale = np.max(np.abs(ref), axis=1)
    diff = np.max(np.abs(got - ref), axis=1)
    zero = scale == 0
    assert np.all(diff[zero] == 0.0), "rows that are exactly zero in the oracle must be zero"
    if np.all(zero):
        return 0.0
    return float(np.max(diff[~zero] / scale[~zero]))


def norm_error(got, ref) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    s = np.max(np.abs(ref))
    return float(np.max(np.abs(got - ref)) / s) if s > 0 else float(np.max(np.abs(got)))
