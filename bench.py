#!/usr/bin/env python3
"""Throughput of the sparse basis convolution's hot path on one MI355X.

One step = neighbour search -> forward (basis evaluated inside) -> transpose
-> backward (dF and dW) over one batch of synthetic input already resident in
HBM.  Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--order auto]

The reported value is neighbour edges per second of whole steps.  Every
kernel of the step is timed with HIP events recorded on its launch stream
(the library's trace hook); the roofline object describes the kernel with
the largest share of the step.  The CPU oracle is timed on this host's cores
on the same workload, outside the timed region.
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "neighbour-edges/s and achieved HBM GB/s (SpMM) + MFMA TFLOP/s, fwd+bwd"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
MFMA_PEAK_TFLOPS = {"f32": 157.3, "bf16": 2500.0}

DESCRIPTIONS = {
    "sphere_1024": "1 cloud, 1024 points on the unit sphere -> first 256; r 0.2, cap 16; "
                   "M 4 monomials x (1-|u|^2)^2; 16 -> 32 channels fp32",
    "ellipsoids_inplace": "32 clouds x 1024 points on ellipsoid surfaces, in place; r 0.1, "
                          "cap 32; M 8; 64 -> 64 channels fp32",
    "ellipsoids_down": "32 clouds x 1024 -> 256 farthest points; r 0.2, cap 32; M 8; "
                       "64 -> 128 channels fp32",
    "events_300k": "300k events, 128x128 pixels, 100 ms uniform; 3x3 block, 10 ms window; "
                   "M 8; 32 -> 32 channels fp32",
    "events_1m_bf16": "1M bursty events, 346x260 pixels, 200 ms; 3x3 block, 5 ms window; M 8; "
                      "64 -> 64 channels bf16 in, fp32 accumulate",
}


def kernel_table(kind, plan, n_in, n_out, E, M, ci, co, sf, blocks_bwd=256):
    """Kernels of one step: name -> (launches per step, algorithmic bytes, flops, on MFMA).

    Bytes count every array the kernel must touch once (gathered rows once per
    row, not once per edge); flops count the multiply-adds x 2 of the
    contraction (MFMA) or of the gather (vector ALU, reported but not a roof).
    """
    geo = 12 * (n_in + n_out) if kind == "points" else 12 * n_in
    W = M * ci * co * sf
    t = {}
    if kind == "points":
        t["points_count"] = (1, 12 * n_out + 16 * n_in + 4 * n_out, 0, False)
        t["points_fill"] = (1, 12 * n_out + 16 * n_in + 8 * n_out + 4 * E, 0, False)
    else:
        t["events_count"] = (1, 24 * n_in, 0, False)
        t["events_fill"] = (1, 28 * n_in + 4 * E, 0, False)
    t["transpose_sort"] = (1, 4 * (n_in + 1) + 16 * E, 0, False)
    basis_launches = 0
    csr_b = 4 * (n_out + 1) + 4 * E + 4 * E * M
    csc_b = 4 * (n_in + 1) + 8 * E + 4 * E * M
    if plan["forward_fused"]:
        t["fwd_fused"] = (1, 4 * (n_out + 1) + 4 * E + geo + n_in * ci * sf + W + 4 * n_out * co,
                          2 * n_out * M * ci * co, True)
    elif plan["forward_order"] == "spmm_first":
        basis_launches += 1
        G = 4 * n_out * M * ci
        t["fwd_spmm"] = (1, csr_b + n_in * ci * sf + G, 2 * E * M * ci, False)
        t["fwd_gemm"] = (1, G + W + 4 * n_out * co, 2 * n_out * M * ci * co, True)
    else:
        basis_launches += 1
        H = 4 * n_in * M * co
        t["fwd_gemm_h"] = (1, n_in * ci * sf + W + H, 2 * n_in * ci * M * co, True)
        t["fwd_spmm_contract"] = (1, csr_b + H + 4 * n_out * co, 2 * E * M * co, False)
    if plan["backward_fused"]:
        part = 4 * blocks_bwd * ci * M * co
        t["bwd_fused"] = (1, 4 * (n_in + 1) + 4 * E + geo + n_out * co * sf + n_in * ci * sf
                          + W + 4 * n_in * ci + part, 4 * n_in * M * ci * co, True)
        t["bwd_dw_reduce"] = (1, part + 4 * M * ci * co, 0, False)
    elif plan["backward_order"] == "spmm_first":
        basis_launches += 1
        D = 4 * n_in * M * co
        t["bwd_spmm_t_expand"] = (1, csc_b + n_out * co * sf + D, 2 * E * M * co, False)
        t["bwd_gemm_df"] = (1, D + W + 4 * n_in * ci, 2 * n_in * M * co * ci, True)
        t["bwd_gemm_dw_t"] = (1, n_in * ci * sf + D + 4 * M * ci * co, 2 * n_in * ci * M * co,
                              True)
    else:
        basis_launches += 1
        G = 4 * n_out * M * ci
        t["bwd_spmm"] = (1, csr_b + n_in * ci * sf + G, 2 * E * M * ci, False)
        t["bwd_gemm_dw"] = (1, G + n_out * co * sf + 4 * M * ci * co, 2 * n_out * M * ci * co,
                            True)
        t["bwd_gemm_dg"] = (1, n_out * co * sf + W + G, 2 * n_out * M * ci * co, True)
        t["bwd_spmm_t"] = (1, csc_b + G + 4 * n_in * ci, 2 * E * M * ci, False)
    if basis_launches:
        t["basis"] = (basis_launches, 4 * (n_out + 1) + 4 * E + geo + 4 * E * M, 0, False)
    return t


def cpu_baseline(w, reps):
    """The oracle on the whole workload: neighbours, basis, forward, transpose, backward."""
    import oracle
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # threadpoolctl missing: report the OpenMP count only
        blas = 1
    times, E = [], 0
    for _ in range(reps):
        t0 = time.perf_counter()
        if w["kind"] == "points":
            rp, ci = oracle.points_csr(w["x_in"], w["in_splits"], w["x_out"], w["out_splits"],
                                       w["radius"], w["k_cap"])
            v = oracle.basis.point_basis(w["x_in"], w["x_out"], rp, ci, w["radius"], w["M"])
        else:
            rp, ci = oracle.events_csr(w["px"], w["py"], w["t"], w["window"], 1, w["width"],
                                       w["height"])
            v = oracle.basis.event_basis(w["px"], w["py"], w["t"], rp, ci, w["tau"])
        oracle.conv.forward(rp, ci, v, w["F"], w["W"])
        oracle.csr_transpose(rp, ci, w["n_in"])
        oracle.conv.backward(rp, ci, v, w["F"], w["W"], w["dY"], w["n_in"])
        times.append(time.perf_counter() - t0)
        E = len(ci)
    med = statistics.median(times)
    return {"value": E / med, "unit": "edges/s", "cores": max(oracle.max_threads(), blas),
            "kind": "oracle",
            "sample": f"whole workload ({E} edges): neighbours, basis, forward, transpose, "
                      f"backward in float64; median of {reps} passes, {med:.2f} s each"}


def graph_timing(step, a, torch):
    """ms per step of HIP-graph replays of one captured step, and the wall time."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for _ in range(2):
            step()
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for _ in range(a.warmup):
        graph.replay()
    torch.cuda.synchronize()
    t_start = torch.cuda.Event(enable_timing=True)
    t_stop = torch.cuda.Event(enable_timing=True)
    wall0 = time.perf_counter()
    t_start.record()
    for _ in range(a.steps):
        graph.replay()
    t_stop.record()
    torch.cuda.synchronize()
    return t_start.elapsed_time(t_stop) / a.steps, time.perf_counter() - wall0


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="ellipsoids_inplace", choices=sorted(DESCRIPTIONS))
    ap.add_argument("--order", default="auto", choices=["auto", "spmm_first", "gemm_first"])
    ap.add_argument("--cpu-reps", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graph", action="store_true",
                    help="time eager steps only (for counter collection, which serialises)")
    ap.add_argument("--copy-probe-mb", type=int, default=0,
                    help="after timing, run one plain device copy of this many MiB "
                         "(calibrates profiler byte counters)")
    a = ap.parse_args(argv)
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if a.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the hot path is built and timed on a single MI355X; "
              "multi-GPU sharding is described in DESIGN.md but not run", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import paper_2012_01170_amd as sbc
    import workloads
    from paper_2012_01170_amd import _lib

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = workloads.WORKLOADS[a.workload]()
    T = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(dev)
    if w["dtype"] == "bf16":
        feat = lambda k: T(w[k + "_bits"].view(np.int16)).view(torch.bfloat16)
        sf = 2
    else:
        feat = lambda k: T(w[k])
        sf = 4
    F, W, dY = feat("F"), feat("W"), feat("dY")
    M, ci, co = w["M"], w["C_in"], w["C_out"]
    if w["kind"] == "points":
        x_in, x_out = T(w["x_in"]), T(w["x_out"])
        s_in, s_out = T(w["in_splits"]), T(w["out_splits"])
        geo = sbc.Geometry(w["basis"], radius=w["radius"], x_in=x_in, x_out=x_out)

        def search():
            return sbc.neighbour_search_points(x_in, s_in, x_out, s_out, w["radius"],
                                               w["k_cap"], sync=False)
    else:
        px, py, tt = T(w["px"]), T(w["py"]), T(w["t"])
        geo = sbc.Geometry("event8", tau=w["tau"], px=px, py=py, t=tt)
        cap = sbc.neighbour_search_events(px, py, tt, w["width"], w["height"], w["window"]).nnz

        def search():
            return sbc.neighbour_search_events(px, py, tt, w["width"], w["height"], w["window"],
                                               col_capacity=cap, sync=False)

    n_in, n_out = w["n_in"], w["n_out"]
    csr0 = search()
    torch.cuda.synchronize()
    E = int(csr0.row_ptr[-1].item())
    plan = sbc.conv_plan(n_out, n_in, csr0.nnz, M, ci, co, F.dtype, a.order)

    def step():
        csr = search()
        Y = sbc.conv_forward(csr, F, W, geometry=geo, order=a.order)
        csc = sbc.csr_transpose(csr)
        dF, dW = sbc.conv_backward(csr, csc, F, W, dY, geometry=geo, order=a.order)
        return Y, dF, dW

    n_cus = torch.cuda.get_device_properties(dev).multi_processor_count
    tr_bwd = 64 if M * co * sf * 64 <= 65536 else 32     # the fused backward's tile rows
    blocks_bwd = max(1, min(256, n_cus, (n_in + tr_bwd - 1) // tr_bwd))
    table = kernel_table(w["kind"], plan, n_in, n_out, E, M, ci, co, sf, blocks_bwd)
    L = _lib.lib()
    # one (start, stop) event pair per kernel per timed step; record once so the
    # underlying HIP events exist before the library records them again
    ev = [{k: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for k in table} for _ in range(a.steps)]
    for d in ev:
        for s0, s1 in d.values():
            s0.record()
            s1.record()

    for _ in range(a.warmup):
        step()
    torch.cuda.synchronize()

    # (1) eager steps with every kernel bracketed by HIP events (trace hook)
    t_start = torch.cuda.Event(enable_timing=True)
    t_stop = torch.cuda.Event(enable_timing=True)
    t_start.record()
    for s in range(a.steps):
        for k, (s0, s1) in ev[s].items():
            _lib.check(L.sbc_trace_kernel(k.encode(), s0.cuda_event, s1.cuda_event))
        step()
    t_stop.record()
    torch.cuda.synchronize()
    L.sbc_trace_clear()
    eager_ms = t_start.elapsed_time(t_stop) / a.steps

    # (2) the same step captured once in a HIP graph (it never synchronises
    # with the host), then replayed: the timed region
    if a.no_graph:
        ms, wall = eager_ms, float("nan")
    else:
        ms, wall = graph_timing(step, a, torch)
    if a.copy_probe_mb > 0:
        src = torch.ones(a.copy_probe_mb << 18, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    kernels = {}
    for k, (launches, nbytes, flops, mfma) in table.items():
        us = statistics.mean(ev[s][k][0].elapsed_time(ev[s][k][1]) for s in range(a.steps)) * 1e3
        kernels[k] = {"us": round(us, 2), "launches": launches,
                      "GB_s": round(nbytes / (us * 1e-6) / 1e9, 1),
                      "TFLOP_s": round(flops / (us * 1e-6) / 1e12, 3) if flops else 0.0}
    dom = max(kernels, key=lambda k: kernels[k]["us"] * kernels[k]["launches"])
    _, nbytes, flops, mfma = table[dom]
    dt = w["dtype"]
    us = kernels[dom]["us"]
    if mfma and flops / (MFMA_PEAK_TFLOPS[dt] * 1e12) > nbytes / (HBM_PEAK_GBS * 1e9):
        achieved, peak, unit, bound = flops / (us * 1e-6) / 1e12, MFMA_PEAK_TFLOPS[dt], "TFLOP/s", "mfma"
    else:
        achieved, peak, unit, bound = nbytes / (us * 1e-6) / 1e9, HBM_PEAK_GBS, "GB/s", "hbm"
    roof = {"bound": bound, "kernel": dom, "achieved": round(achieved, 3), "peak": peak,
            "unit": unit, "frac": round(achieved / peak, 4), "traffic": None,
            "per_launch": {"bytes": nbytes, "flops": flops, "us": us}}

    out = {"metric": METRIC, "value": E / (ms * 1e-3), "unit": "edges/s", "n_gpus": 1,
           "steps": a.steps, "warmup": a.warmup, "ms_per_step": round(ms, 4),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": dt,
           "data": "synthetic (seeded generators; inputs resident in HBM)",
           "config": {"workload": f"{a.workload}: {DESCRIPTIONS[a.workload]}", "n_in": n_in,
                      "n_out": n_out, "edges": E, "M": M, "C_in": ci, "C_out": co,
                      "plan": plan,
                      "timing": "eager steps" if a.no_graph else "HIP graph replays of the captured step",
                      "eager_ms_per_step": round(eager_ms, 4), "wall_s": round(wall, 3)},
           "roofline": roof, "kernels": kernels}
    if not a.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, a.cpu_reps)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
