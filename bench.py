#!/usr/bin/env python3
"""Throughput of the sparse basis convolution's hot path on one MI355X.

One step = neighbour search -> forward (basis evaluated inside) -> transpose
-> backward (dF and dW) over one batch of synthetic input already resident in
HBM (for event streams the transpose comes out of the search itself, by the
reverse search over the same pixel lists).  Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--order auto]

The reported value is neighbour edges per second of whole steps.  Every
kernel of the step is timed with HIP events recorded on its launch stream
(the library's trace hook); the roofline object describes the kernel with
the largest share of the step.  The CPU oracle is timed on this host's cores
on the same workload, outside the timed region.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import re
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
    "ellipsoids_weighted": "32 clouds x 1024 points on ellipsoid surfaces, in place; r 0.1, "
                           "cap 32; weighted convolution (Eq. 11), M 10 monomials up to 2nd "
                           "order; 64 -> 64 channels fp32",
    "ellipsoids_featureless": "32 clouds x 1024 points on ellipsoid surfaces, in place; r 0.1, "
                              "cap 32; featureless convolution (Eq. 9-10) with the weighted "
                              "M 10 basis; 32 output channels fp32",
    "events_300k_decays2": "300k events, 128x128 pixels, 100 ms uniform; 3x3 block, 10 ms "
                           "window; learned decays, 2 per offset (M 16), with their gradient; "
                           "32 -> 32 channels fp32",
    "ellipsoids_sampling": "32 clouds x 1024 points on ellipsoid surfaces; uncapped in-place "
                           "ball r 0.1, then rejection sampling and approximate farthest points "
                           "up to 256 per cloud",
    "table2_flexconv": "the paper's Table 2 operator shape: 8 clouds x 4096 points in the unit "
                       "cube, in place, the 9 nearest within r 0.25 (E 294,912); M 4; 64 -> 64 "
                       "channels fp32; forward, transpose and backward, the search left out as "
                       "in the table",
    "events_stream": "300k events, 128x128 pixels, 100 ms uniform, through the deployment form "
                     "(per-pixel decayed sums, Eq. 13-15) in batches of 4096; tau 10 ms; "
                     "32 -> 32 channels fp32",
    "events_300k_lif": "300k events, 128x128 pixels, 100 ms uniform -> the 64x64 stream by "
                       "leaky integrate-and-fire: 3x3 fields, stride 2, decay 4 ms, threshold "
                       "1.6, reset -3; float64 potentials",
}


SRC_DIR = os.path.join(ROOT, "paper_2012_01170_amd", "csrc")
PROFILES = os.path.join(ROOT, "profiles")
# device function -> the name the library's trace hook gives its launch
TRACE_NAME = {"bwd_ws_kernel": "bwd_fused", "fwd_fused_kernel": "fwd_fused",
              "fwd_reg_kernel": "fwd_fused", "fwd_onehot_kernel": "fwd_fused",
              "dw_reduce_kernel": "bwd_dw_reduce",
              "sample_kernel<true>": "sample", "sample_kernel<false>": "sample_count",
              "lif_cell_kernel": "lif_cells", "lif_emit_kernel": "lif_emit",
              "stream_gather_kernel": "stream_gather", "stream_update_kernel": "stream_update"}


def trace_name(kernel):
    """The trace-hook name of a profiled kernel ('f<args>'), or None."""
    if kernel in TRACE_NAME:
        return TRACE_NAME[kernel]
    base = kernel.split("<")[0]
    if base == "bwd_ws_kernel":  # <M, CI, CO, basis, ...>: basis 16 is the decay derivative
        args = kernel[len(base) + 1:].split(",")
        return "decay_fused" if len(args) > 3 and args[3].strip() == "16" else "bwd_fused"
    if base == "featureless_kernel":  # <M, mode, writes Z>
        return "featureless_fwd" if kernel.rstrip(">").endswith("true") else "featureless_rowsum"
    if base == "spmm_kernel":  # <M, contract, X type>: named by direction, see SPMM_DIRECTION
        args = kernel[len(base) + 1:].split(",")
        return "spmm_contract" if len(args) > 1 and args[1].strip() == "true" else "spmm_expand"
    return TRACE_NAME.get(base)


# The generic gather kernel serves several launches; each workload's step has
# at most one launch per direction, so its counters are filed by direction.
SPMM_DIRECTION = {"fwd_spmm": "spmm_expand", "bwd_spmm": "spmm_expand",
                  "bwd_spmm_t_expand": "spmm_expand", "decay_spmm": "spmm_expand",
                  "fwd_spmm_contract": "spmm_contract", "bwd_spmm_t": "spmm_contract"}


def source_fingerprint():
    """Hash of the HIP sources: byte counts taken on other sources do not apply."""
    h = hashlib.sha256()
    for name in sorted(os.listdir(SRC_DIR)):
        if name.endswith((".hip", ".hpp")):
            h.update(name.encode())
            with open(os.path.join(SRC_DIR, name), "rb") as f:
                h.update(f.read())
    return h.hexdigest()[:16]


def kernel_fingerprint(base):
    """Hash of the HIP source that defines device function `base` and of the
    shared headers: a kernel's byte counts stay valid while these are unchanged."""
    h = hashlib.sha256()
    names = sorted(os.listdir(SRC_DIR))
    pat = re.compile(r"\b" + re.escape(base) + r"\s*\(")
    for name in names:
        path = os.path.join(SRC_DIR, name)
        if name.endswith(".hpp") or (name.endswith(".hip") and pat.search(open(path).read())):
            h.update(name.encode())
            with open(path, "rb") as f:
                h.update(f.read())
    return h.hexdigest()[:16]


def short_kernel_name(name):
    """'void ns::(anonymous namespace)::f<...>(args)' -> 'f<...>'."""
    name = name.replace("(anonymous namespace)::", "")
    if name.startswith("void "):
        name = name[5:]
    depth, cut = 0, len(name)
    for i, ch in enumerate(name):
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            cut = i
            break
    return name[:cut].split("::")[-1] if "<" not in name[:cut] else \
        name[:cut][name[:cut].rfind("::", 0, name[:cut].find("<")) + 2:]


def read_traffic(workload):
    """HBM bytes per dispatch of each traced kernel from a committed counter summary.

    Returns (table, note): table maps trace name -> bytes per launch for the
    kernels whose source (kernel_fingerprint) is unchanged since the counters
    were taken; None when there is no summary.
    """
    path = os.path.join(PROFILES, f"hbm_traffic_{workload}.txt")
    if not os.path.exists(path):
        return None, "no counter summary"
    table, stale = {}, []
    with open(path) as f:
        for line in f:
            parts = line.split()
            if len(parts) >= 7 and parts[0] == "traffic":
                if parts[6] == kernel_fingerprint(parts[2]):
                    table[parts[1]] = float(parts[5])
                else:
                    stale.append(parts[1])
    note = os.path.basename(path)
    if stale:
        note += " (changed since the counters were taken: " + ", ".join(stale) + ")"
    return table, note


def _counter_rows(directory):
    files = glob.glob(os.path.join(directory, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {directory}")
    with open(files[0]) as f:
        return list(csv.DictReader(f))


def summarize_traffic(fetch_dir, write_dir, probe_mb, command):
    """Text summary of FETCH_SIZE / WRITE_SIZE per dispatch, scaled by a copy probe.

    The probe is one plain device-to-device copy of probe_mb MiB run by the
    profiled command after its steps: it reads and writes exactly that many
    bytes, so true bytes / counter bytes calibrates each counter.
    """
    probe_kib = probe_mb * 1024.0
    out = [f"# HBM traffic per dispatch from rocprofv3 byte counters", f"# command: {command}",
           f"source_fingerprint: {source_fingerprint()}"]
    per = {}
    factors = {}
    for counter, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        rows = [r for r in _counter_rows(d) if r["Counter_Name"] == counter]
        copies = [float(r["Counter_Value"]) for r in rows if "copyBuffer" in r["Kernel_Name"]]
        probe = max(copies) if copies else 0.0
        if probe <= 0.0:
            raise SystemExit(f"{counter}: no copy-probe dispatch found in {d}")
        factors[counter] = probe_kib / probe
        out.append(f"{counter.lower()}_factor: {factors[counter]:.4f}  "
                   f"(copy probe {probe_mb} MiB; counter read {probe:.0f} KiB)")
        for r in rows:
            k = short_kernel_name(r["Kernel_Name"])
            per.setdefault(k, {}).setdefault(counter, []).append(float(r["Counter_Value"]))
    out.append("# kernel  dispatches  FETCH_KiB/dispatch  WRITE_KiB/dispatch  "
               "scaled bytes/dispatch")
    rows_out = []
    for k, c in per.items():
        if "FETCH_SIZE" not in c or "WRITE_SIZE" not in c:
            continue
        fk = statistics.mean(c["FETCH_SIZE"])
        wk = statistics.mean(c["WRITE_SIZE"])
        b = (fk * factors["FETCH_SIZE"] + wk * factors["WRITE_SIZE"]) * 1024.0
        rows_out.append((b, k, len(c["FETCH_SIZE"]), fk, wk))
    for b, k, n, fk, wk in sorted(rows_out, reverse=True):
        out.append(f"kernel {k}  {n}  {fk:.1f}  {wk:.1f}  {b:.0f}")
    # one line per traced launch name, the form bench.py reads back
    for b, k, n, fk, wk in sorted(rows_out, reverse=True):
        base = k.split("<")[0]
        if trace_name(k):
            out.append(f"traffic {trace_name(k)} {base} {fk:.1f} {wk:.1f} {b:.0f} "
                       f"{kernel_fingerprint(base)}")
    return "\n".join(out) + "\n"


def _counter_by_kernel(directory, counter):
    """Per profiled kernel (short name): the list of one counter's readings
    over its dispatches, and the largest reading of a copy kernel (the probe)."""
    per, probe = {}, 0.0
    for r in _counter_rows(directory):
        if r["Counter_Name"] != counter:
            continue
        if "copyBuffer" in r["Kernel_Name"]:
            probe = max(probe, float(r["Counter_Value"]))
            continue
        per.setdefault(short_kernel_name(r["Kernel_Name"]), []).append(float(r["Counter_Value"]))
    return per, probe


def summarize_route(workload, runs, probe_mb, command, steps):
    """Side-by-side summary of the evaluation orders of one workload (Table 1's
    two orders): per order, the graph-timed step and its kernels' HIP-event
    times, then per profiled kernel its dispatches per step, HBM bytes per
    dispatch (FETCH_SIZE + WRITE_SIZE scaled by the copy probe) and MFMA-busy
    cycles per dispatch (summed over SIMDs), and the step's totals.
    runs: order -> (bench json, fetch dir, write dir, mfma dir); steps: the
    profiled runs' step count (warm-up included)."""
    out = ["# evaluation orders compared on one workload: step time, kernel times, HBM bytes "
           "and MFMA-busy cycles",
           "# (dispatches per step count the profiled run's warm-up and timed steps; the "
           "search also runs twice while the benchmark is set up)", f"# command: {command}",
           f"source_fingerprint: {source_fingerprint()}", f"workload: {workload}"]
    for order, (bj, fdir, wdir, mdir) in runs.items():
        with open(bj) as f:
            b = json.loads([l for l in f if l.startswith("{")][-1])
        fetch, probe_f = _counter_by_kernel(fdir, "FETCH_SIZE")
        write, probe_w = _counter_by_kernel(wdir, "WRITE_SIZE")
        mfma, _ = _counter_by_kernel(mdir, "SQ_VALU_MFMA_BUSY_CYCLES")
        ff = probe_mb * 1024.0 / probe_f if probe_f else float("nan")
        wf = probe_mb * 1024.0 / probe_w if probe_w else float("nan")
        out.append(f"order {order}: plan {b['config']['plan']}; step {b['ms_per_step'] * 1e3:.1f} us "
                   f"(graph replays)")
        out.append("#   trace name  us  launches")
        for k, v in b["kernels"].items():
            out.append(f"  {order} time {k} {v['us']:.1f} {v['launches']}")
        out.append("#   profiled kernel  dispatches_per_step  HBM_MB_per_dispatch  "
                   "MFMA_busy_Mcycles_per_dispatch")
        tot_b = tot_m = 0.0
        for k in sorted(fetch, key=lambda k: -sum(fetch[k])):
            if k not in write or k.startswith("vectorized_elementwise"):
                continue  # torch's own fill of the copy probe
            n = len(fetch[k])
            mb = (statistics.mean(fetch[k]) * ff + statistics.mean(write[k]) * wf) * 1024.0 / 1e6
            mc = statistics.mean(mfma[k]) / 1e6 if k in mfma else 0.0
            per_step = n / steps
            tot_b += mb * per_step
            tot_m += mc * per_step
            if mb * per_step >= 0.5 or mc > 0:
                out.append(f"  {order} counters {k} {per_step:g} {mb:.1f} {mc:.2f}")
        out.append(f"  {order} step_total HBM_MB {tot_b:.1f} MFMA_busy_Mcycles {tot_m:.2f}")
    return "\n".join(out) + "\n"


def summarize_counters(dirs, command):
    """Text summary of rocprofv3 --pmc runs of SQ counters: per profiled kernel
    (those with at least 2% of the largest one's wave-cycles), each counter's
    reading per dispatch
    (summed over the chip as the profiler reports it), averaged over the
    dispatches."""
    per = {}
    for d in dirs:
        for r in _counter_rows(d):
            k = short_kernel_name(r["Kernel_Name"])
            per.setdefault(k, {}).setdefault(r["Counter_Name"], {}).setdefault(
                r.get("Dispatch_Id", ""), 0.0)
            per[k][r["Counter_Name"]][r.get("Dispatch_Id", "")] += float(r["Counter_Value"])
    out = ["# rocprofv3 SQ counters per dispatch (mean over dispatches)", f"# command: {command}",
           f"source_fingerprint: {source_fingerprint()}"]
    def weight(k):
        return statistics.mean(per[k].get("SQ_WAVE_CYCLES", {"": 0.0}).values())

    order = sorted(per, key=lambda k: -weight(k))
    top = weight(order[0]) if order else 0.0
    for k in order:
        cs = per[k]
        if "SQ_WAVE_CYCLES" not in cs or weight(k) < 0.02 * top:
            continue  # kernels below 2% of the largest one's wave-cycles are left out
        out.append(f"kernel {k}")
        for c in sorted(cs):
            vals = list(cs[c].values())
            out.append(f"  {c} {statistics.mean(vals):.4g}  ({len(vals)} dispatches)")
    return "\n".join(out) + "\n"


def summarize_trace(trace_dir, command, bench_json=None):
    """Text summary of a rocprofv3 --kernel-trace --stats run (top kernels by time)."""
    files = glob.glob(os.path.join(trace_dir, "**", "*kernel_stats.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no kernel_stats.csv under {trace_dir}")
    with open(files[0]) as f:
        rows = list(csv.DictReader(f))
    out = ["# rocprofv3 kernel statistics", f"# command: {command}",
           f"source_fingerprint: {source_fingerprint()}",
           "# calls  total_us  avg_us  min_us  max_us  share%  kernel"]
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        out.append(f"{int(r['Calls']):6d}  {float(r['TotalDurationNs']) / 1e3:10.1f}  "
                   f"{float(r['AverageNs']) / 1e3:8.2f}  {float(r['MinNs']) / 1e3:8.2f}  "
                   f"{float(r['MaxNs']) / 1e3:8.2f}  {float(r['Percentage']):5.2f}  "
                   f"{short_kernel_name(r['Name'])}")
    if bench_json:
        with open(bench_json) as f:
            line = [l for l in f if l.startswith("{")][-1]
        b = json.loads(line)
        out.append("# the same run's bench line: HIP-event time per launch (trace hook)")
        for k, v in b["kernels"].items():
            out.append(f"bench {k} {v['us']} us")
        r = b["roofline"]
        out.append(f"bench roofline {r['kernel']} {r['bound']} achieved {r['achieved']} "
                   f"{r['unit']} frac {r['frac']}")
    return "\n".join(out) + "\n"


def sampling_table(n, E, n_batch):
    """Kernels of one sampling step (uncapped ball search, rejection sampling
    and approximate farthest points): name -> (launches, bytes, flops, MFMA)."""
    return {
        "points_count": (1, 12 * n + 16 * n + 4 * n, 0, False),
        "points_fill": (1, 12 * n + 16 * n + 8 * n + 4 * E, 0, False),
        "sample_count": (1, 4 * (n_batch + 1) + 4 * (n + 1) + 4 * E + 12 * n, 0, False),
        "sample": (1, 4 * (n_batch + 1) + 4 * (n + 1) + 4 * E + 12 * n + 8 * n, 0, False),
    }


def lif_table(n, npix, slots, spikes):
    """Kernels of one LIF step (pixel lists, the cells, the emission): name ->
    (launches, algorithmic bytes, flops, MFMA).  lif_sort spans the key,
    sort, bounds and time kernels and the flag clear."""
    return {
        "lif_sort": (1, 12 * n + 8 * n + 4 * (npix + 1) + 4 * n * slots, 0, False),
        "lif_cells": (1, 4 * (npix + 1) + 8 * n + 4 * spikes, 0, False),
        "lif_emit": (1, 8 * n * slots + 12 * spikes + 16 * spikes, 0, False),
    }


def stream_table(B, npix, C, P):
    """Kernels of one batch of the deployment form (each runs once per batch):
    name -> (launches per batch, algorithmic bytes, flops, MFMA)."""
    lists = 12 * B + 8 * B + 4 * (npix + 1)
    return {
        "stream_lists": (1, lists, 0, False),
        "stream_gather": (1, lists + 4 * npix + 4 * npix * C + 4 * B * C + 4 * B * 8 * C, 0,
                          False),
        "stream_gemm": (1, 4 * B * 8 * C + 4 * 8 * C * P + 4 * B * P, 2 * B * 8 * C * P, True),
        "stream_update": (1, 4 * (npix + 1) + 8 * B + 4 * B * C + 8 * npix * C + 8 * npix, 0,
                          False),
    }


def featureless_table(n_in, n_out, E, M, P):
    """Kernels of one featureless step (search, Z = G~ Phi, dPhi = G~^T dZ):
    name -> (launches, algorithmic bytes, flops, on MFMA)."""
    geo = 12 * (n_in + n_out)
    rows = 4 * (n_out + 1) + 4 * E + geo
    return {
        "points_count": (1, 12 * n_out + 16 * n_in + 4 * n_out, 0, False),
        "points_fill": (1, 12 * n_out + 16 * n_in + 8 * n_out + 4 * E, 0, False),
        "featureless_fwd": (1, rows + 4 * M * P + 4 * n_out * P, 2 * n_out * M * P, False),
        "featureless_rowsum": (1, rows + 4 * n_out * M, 0, False),
        "featureless_dphi": (1, 4 * n_out * M + 4 * n_out * P + 4 * M * P, 2 * n_out * M * P,
                             True),
    }


def kernel_table(kind, plan, n_in, n_out, E, M, ci, co, sf, blocks_bwd=256, npix=0):
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
        # pixel tiles: list bounds and lists (index, time) in; the row and
        # column lengths out, or the row and column bounds in and the rows
        # and columns of both patterns out
        t["events_count"] = (1, 4 * (npix + 1) + 8 * n_in + 8 * n_in, 0, False)
        t["events_fill"] = (1, 4 * (npix + 1) + 8 * n_in + 8 * (n_in + 1) + 8 * E, 0, False)
    if kind == "points":
        # block-diagonal transpose, one workgroup per cloud: row bounds and
        # column indices in, column bounds, rows and edge positions out
        t["transpose_batched"] = (1, 4 * (n_out + 1) + 4 * E + 4 * (n_in + 1) + 8 * E, 0, False)
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
        # compulsory bytes only: the per-block dW partials the kernel writes
        # for the ordered reduction are its own scratch, not algorithmic
        # traffic (the byte counters show them)
        t["bwd_fused"] = (1, 4 * (n_in + 1) + 4 * E + geo + n_out * co * sf + n_in * ci * sf
                          + W + 4 * n_in * ci, 4 * n_in * M * ci * co, True)
        t["bwd_dw_reduce"] = (1, 4 * M * ci * co, 0, False)
    elif plan["backward_order"] == "spmm_first":
        basis_launches += 1
        D = 4 * n_in * M * co
        t["bwd_spmm_t_expand"] = (1, csc_b + n_out * co * sf + D, 2 * E * M * co, False)
        t["bwd_gemm_df"] = (1, D + W + 4 * n_in * ci, 2 * n_in * M * co * ci, True)
        t["bwd_gemm_dw_t"] = (1, n_in * ci * sf + D + 4 * M * ci * co, 2 * n_in * ci * M * co,
                              True)
    else:
        # an event stream's transpose comes from the search without edge
        # positions: the transposed entries' values are evaluated once more
        basis_launches += 2 if kind == "events" else 1
        G = 4 * n_out * M * ci
        t["bwd_spmm"] = (1, csr_b + n_in * ci * sf + G, 2 * E * M * ci, False)
        t["bwd_gemm_dw"] = (1, G + n_out * co * sf + 4 * M * ci * co, 2 * n_out * M * ci * co,
                            True)
        t["bwd_gemm_dg"] = (1, n_out * co * sf + W + G, 2 * n_out * M * ci * co, True)
        t["bwd_spmm_t"] = (1, csc_b + G + 4 * n_in * ci, 2 * E * M * ci, False)
    if basis_launches:
        t["basis"] = (basis_launches, 4 * (n_out + 1) + 4 * E + geo + 4 * E * M, 0, False)
    return t


def _blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # threadpoolctl missing: report the OpenMP count only
        return 1


def event_prefix(w, n_events):
    """The first n_events of an event workload: a stream of its own whose
    pattern is exactly the first n_events rows of the whole one (an event's
    neighbours all come before it), so its timings are a bounded sample of
    the same work."""
    if n_events >= w["n_in"]:
        return w, w["n_in"]
    v = dict(w)
    for k in ("px", "py", "t", "F", "dY"):
        v[k] = w[k][:n_events]
    v["n_in"] = v["n_out"] = n_events
    return v, n_events


def oracle_stages(w):
    """One pass of the oracle over workload w, stage by stage: (seconds per
    stage, edge count)."""
    import oracle
    st = {}
    in_step = w.get("search_in_step", True)
    t0 = time.perf_counter()
    if w["kind"] == "points":
        rp, ci = oracle.points_csr(w["x_in"], w["in_splits"], w["x_out"], w["out_splits"],
                                   w["radius"], w["k_cap"])
    else:
        rp, ci = oracle.events_csr(w["px"], w["py"], w["t"], w["window"], 1, w["width"],
                                   w["height"])
    t1 = time.perf_counter()
    if in_step:
        st["neighbours"] = t1 - t0
    if w["kind"] == "points":
        v = oracle.basis.point_values(w["basis"], w["x_in"], w["x_out"], rp, ci, w["radius"],
                                      w["M"])
    else:
        v = oracle.basis.event_values(w["basis"], w["px"], w["py"], w["t"], rp, ci, w["tau"],
                                      w.get("decays"))
    t2 = time.perf_counter()
    st["basis"] = t2 - t1
    if w.get("sampling"):
        smp = w["sampling"]
        oracle.sampling.approx_ifp_after_rejection(w["x_in"], w["in_splits"], smp["per_cloud"],
                                                   rp, ci)
        st["sampling"] = time.perf_counter() - t2
        return st, len(ci)
    if w.get("featureless"):
        Phi = w["W"][:, 0, :]
        oracle.conv.featureless_forward(rp, ci, v, Phi)
        t3 = time.perf_counter()
        oracle.conv.featureless_backward(rp, ci, v, w["dY"])
        st["forward"], st["backward"] = t3 - t2, time.perf_counter() - t3
        return st, len(ci)
    oracle.conv.forward(rp, ci, v, w["F"], w["W"])
    t3 = time.perf_counter()
    oracle.csr_transpose(rp, ci, w["n_in"])
    t4 = time.perf_counter()
    oracle.conv.backward(rp, ci, v, w["F"], w["W"], w["dY"], w["n_in"])
    t5 = time.perf_counter()
    st["forward"], st["transpose"], st["backward"] = t3 - t2, t4 - t3, t5 - t4
    if w["basis"] == "event_decays":
        vd = oracle.basis.event_decay_basis(w["px"], w["py"], w["t"], rp, ci, w["decays"],
                                            derivative=True)
        oracle.conv.decay_backward(rp, ci, vd, w["F"], w["W"], w["dY"])
        st["decay_gradient"] = time.perf_counter() - t5
    return st, len(ci)


def _median_stages(w, reps):
    runs, E = [], 0
    for _ in range(reps):
        st, E = oracle_stages(w)
        runs.append(st)
    stages = {k: statistics.median(r[k] for r in runs) for k in runs[0]}
    total = statistics.median(sum(r.values()) for r in runs)
    return stages, total, E


# events per bounded oracle sample of an event workload (a prefix of the
# stream): about 10-30 s of float64 work on a 16-thread host
ORACLE_EVENT_SAMPLE = 100_000


def cpu_baseline(w, reps):
    """The oracle as written (float64, untuned), timed stage by stage on this
    host's cores: neighbours, basis, forward, transpose, backward.  Point
    workloads run whole, and once more on one thread; event streams run on a
    prefix of ORACLE_EVENT_SAMPLE events."""
    import oracle
    if w["kind"] == "stream":
        t0 = time.perf_counter()
        oracle.conv.deployment_stream(w["px"], w["py"], w["t"], w["F"].astype("float64"),
                                      w["W"].astype("float64"), w["width"], w["height"],
                                      w["tau"])
        sec = time.perf_counter() - t0
        return {"value": w["n_in"] / sec, "unit": "events/s", "cores": 1, "kind": "oracle",
                "sample": f"whole stream ({w['n_in']} events) through the per-event recursion "
                          f"in float64, one pass of {sec:.2f} s"}
    if w["kind"] == "lif":
        times = []
        for _ in range(reps):
            t0 = time.perf_counter()
            out = oracle.sampling.lif(w["px"], w["py"], w["t"], w["width"], w["height"],
                                      w["kernel"], w["stride"], w["decay"], w["v_thresh"],
                                      w["v_reset"])
            times.append(time.perf_counter() - t0)
        med = statistics.median(times)
        return {"value": w["n_in"] / med, "unit": "events/s", "cores": 1, "kind": "oracle",
                "sample": f"whole stream ({w['n_in']} events -> {len(out)}) through the "
                          f"sequential sampler in float64; median of {reps} passes, "
                          f"{med:.2f} s each"}
    if w["kind"] == "events":
        ws, n_s = event_prefix(w, ORACLE_EVENT_SAMPLE)
        what = (f"the first {n_s} of the stream's {w['n_in']} events (a prefix is the same "
                f"pattern's first rows)")
    else:
        ws, what = w, "whole workload"
    stages, total, E = _median_stages(ws, reps)
    cores = max(oracle.max_threads(), _blas_threads())
    steps = ", ".join(stages)
    out = {"value": E / total, "unit": "edges/s", "cores": cores, "kind": "oracle",
           "sample": f"{what}, {E} edges: {steps} in float64; median of {reps} passes, "
                     f"{total:.2f} s each",
           "stages": {k: {"s": round(t, 4), "edges_per_s": round(E / t, 1) if t > 0 else None}
                      for k, t in stages.items()}}
    if w["kind"] == "points":
        try:
            from threadpoolctl import threadpool_limits
        except ImportError:
            threadpool_limits = None
        if threadpool_limits is not None:
            with threadpool_limits(limits=1):
                st1, tot1, _ = _median_stages(ws, reps)
            out["single_thread"] = {
                "value": E / tot1, "unit": "edges/s", "cores": 1,
                "stages": {k: {"s": round(t, 4),
                               "edges_per_s": round(E / t, 1) if t > 0 else None}
                           for k, t in st1.items()}}
    return out


def replay_distribution(graph, steps, torch, flush=None):
    """Per-replay times (ms) of a captured step: each replay bracketed by its
    own events; with `flush`, a write of a 512 MiB buffer runs before each
    bracket, evicting the 256 MB last-level cache (cold inputs)."""
    times = []
    for _ in range(steps):
        if flush is not None:
            flush.fill_(1.0)
        s0 = torch.cuda.Event(enable_timing=True)
        s1 = torch.cuda.Event(enable_timing=True)
        s0.record()
        graph.replay()
        s1.record()
        torch.cuda.synchronize()
        times.append(s0.elapsed_time(s1))
    times.sort()
    q = lambda f: times[min(len(times) - 1, int(round(f * (len(times) - 1))))]
    return {"median_ms": round(statistics.median(times), 4), "p10_ms": round(q(0.1), 4),
            "p90_ms": round(q(0.9), 4), "replays": len(times)}


def measure(a, w, table, step, torch, _lib, dev):
    """Warm-up, eager steps with every kernel bracketed by HIP events (the
    library's trace hook), then HIP-graph replays of the captured step (the
    timed region).  Returns (ms per step, eager ms per step, wall s, the
    per-kernel table, the roofline of the dominant kernel, the single-replay
    distributions hot and cold)."""
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
        ms, wall, dist = eager_ms, float("nan"), None
    else:
        ms, wall, dist = graph_timing(step, a, torch)
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
    traffic, traffic_src = read_traffic(a.workload)
    traffic = traffic.get(SPMM_DIRECTION.get(dom, dom)) if traffic else None
    roof = {"bound": bound, "kernel": dom, "achieved": round(achieved, 3), "peak": peak,
            "unit": unit, "frac": round(achieved / peak, 4),
            "traffic": round(traffic) if traffic is not None else None,
            "per_launch": {"bytes": nbytes, "flops": flops, "us": us,
                           "traffic_over_algorithmic":
                               round(traffic / nbytes, 3) if traffic is not None else None,
                           "traffic_source": traffic_src}}

    return ms, eager_ms, wall, kernels, roof, dist


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
    ms, wall = t_start.elapsed_time(t_stop) / a.steps, time.perf_counter() - wall0
    # the spread of single replays, with the inputs hot in the caches and
    # with the last-level cache evicted before each replay
    dist = {"hot": replay_distribution(graph, a.steps, torch)}
    if not a.no_cold:
        flush = torch.empty(512 << 18, dtype=torch.float32, device=torch.device("cuda:0"))
        dist["cold"] = replay_distribution(graph, a.steps, torch, flush=flush)
        del flush
    return ms, wall, dist


def lif_main(a, w, T, torch, sbc, _lib, dev):
    """One step: the input stream (resident in HBM) through the LIF sampler to
    the next stream, unsynchronised; the value is input events per second."""
    px, py, tt = T(w["px"]), T(w["py"]), T(w["t"])
    args = (px, py, tt, w["width"], w["height"], w["kernel"], w["stride"], w["decay"],
            w["v_thresh"], w["v_reset"])
    spikes = sbc.lif_sample_events(*args)[4]
    nsd = (w["kernel"] - 1) // w["stride"] + 1

    def step():
        return sbc.lif_sample_events(*args, sync=False)

    n = w["n_in"]
    table = lif_table(n, w["width"] * w["height"], nsd * nsd, spikes)
    ms, eager_ms, wall, kernels, roof, dist = measure(a, w, table, step, torch, _lib, dev)
    out = {"metric": "LIF event sampler throughput (input events per second)",
           "value": n / (ms * 1e-3), "unit": "events/s", "n_gpus": 1, "steps": a.steps,
           "warmup": a.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": w["dtype"],
           "data": "synthetic (seeded generators; inputs resident in HBM)",
           "config": {"workload": f"{a.workload}: {DESCRIPTIONS[a.workload]}", "n_in": n,
                      "n_out_events": spikes, "grid": [-(-w["width"] // w["stride"]),
                                                       -(-w["height"] // w["stride"])],
                      "timing": "eager steps" if a.no_graph else "HIP graph replays of the captured step",
                      "eager_ms_per_step": round(eager_ms, 4), "wall_s": round(wall, 3),
                      "replays": dist},
           "roofline": roof, "kernels": kernels}
    if not a.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, a.cpu_reps)
    print(json.dumps(out), flush=True)
    return 0


def stream_main(a, w, T, torch, sbc, _lib, dev):
    """One step: the whole input stream (resident in HBM) through the
    deployment form in batches, the state starting from zero; the value is
    input events per second."""
    px, py, tt, F, W = T(w["px"]), T(w["py"]), T(w["t"]), T(w["F"]), T(w["W"])
    n, B, C, P = w["n_in"], w["batch"], w["C_in"], w["C_out"]
    st = sbc.EventStream(w["width"], w["height"], C, w["tau"], device=dev)

    def step():
        st.z.zero_()
        st.z_time.zero_()
        return [st.step(px[a0:a0 + B], py[a0:a0 + B], tt[a0:a0 + B], F[a0:a0 + B], W)
                for a0 in range(0, n, B)]

    batches = (n + B - 1) // B
    table = {k: (batches, b, f, m) for k, (_, b, f, m) in
             stream_table(B, w["width"] * w["height"], C, P).items()}
    ms, eager_ms, wall, kernels, roof, dist = measure(a, w, table, step, torch, _lib, dev)
    out = {"metric": "deployment-form stream throughput (input events per second)",
           "value": n / (ms * 1e-3), "unit": "events/s", "n_gpus": 1, "steps": a.steps,
           "warmup": a.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": w["dtype"],
           "data": "synthetic (seeded generators; inputs resident in HBM)",
           "config": {"workload": f"{a.workload}: {DESCRIPTIONS[a.workload]}", "n_in": n,
                      "batch": B, "batches": batches, "C_in": C, "C_out": P,
                      "timing": "eager steps" if a.no_graph else "HIP graph replays of the captured step",
                      "eager_ms_per_step": round(eager_ms, 4), "wall_s": round(wall, 3),
                      "replays": dist},
           "roofline": roof, "kernels": kernels}
    if not a.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, a.cpu_reps)
    print(json.dumps(out), flush=True)
    return 0


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="events_300k", choices=sorted(DESCRIPTIONS))
    ap.add_argument("--order", default="auto", choices=["auto", "spmm_first", "gemm_first"])
    ap.add_argument("--cpu-reps", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-cold", action="store_true",
                    help="skip the single replays with the last-level cache evicted")
    ap.add_argument("--no-graph", action="store_true",
                    help="time eager steps only (for counter collection, which serialises)")
    ap.add_argument("--copy-probe-mb", type=int, default=0,
                    help="after timing, run one plain device copy of this many MiB "
                         "(calibrates profiler byte counters)")
    ap.add_argument("--summarize-trace", metavar="DIR",
                    help="print a summary of a rocprofv3 --kernel-trace --stats output and exit")
    ap.add_argument("--summarize-traffic", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="print per-dispatch HBM bytes from two rocprofv3 --pmc outputs and exit")
    ap.add_argument("--bench-json", help="with --summarize-trace: the profiled run's bench line")
    ap.add_argument("--summarize-route", nargs="+", metavar="ARG",
                    help="WORKLOAD then, per order, ORDER BENCH_JSON FETCH_DIR WRITE_DIR MFMA_DIR: "
                         "print the evaluation orders side by side and exit")
    ap.add_argument("--summarize-counters", nargs="+", metavar="DIR",
                    help="print per-kernel means of rocprofv3 --pmc counter runs and exit")
    ap.add_argument("--command", default="", help="the profiled command, quoted in a summary")
    a = ap.parse_args(argv)
    if a.summarize_trace:
        sys.stdout.write(summarize_trace(a.summarize_trace, a.command, a.bench_json))
        return 0
    if a.summarize_counters:
        sys.stdout.write(summarize_counters(a.summarize_counters, a.command))
        return 0
    if a.summarize_route:
        w, rest = a.summarize_route[0], a.summarize_route[1:]
        if len(rest) % 5 or a.copy_probe_mb <= 0:
            ap.error("--summarize-route: WORKLOAD (ORDER JSON FETCH WRITE MFMA)... and "
                     "--copy-probe-mb")
        runs = {rest[i]: tuple(rest[i + 1:i + 5]) for i in range(0, len(rest), 5)}
        sys.stdout.write(summarize_route(w, runs, a.copy_probe_mb, a.command,
                                         a.steps + a.warmup))
        return 0
    if a.summarize_traffic:
        if a.copy_probe_mb <= 0:
            ap.error("--summarize-traffic needs --copy-probe-mb (the probe size of the run)")
        sys.stdout.write(summarize_traffic(*a.summarize_traffic, a.copy_probe_mb, a.command))
        return 0
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if a.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the hot path is built and timed on a single MI355X; "
              "runs on more than one GPU are not made", file=sys.stderr)
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
    if w["kind"] == "lif":
        return lif_main(a, w, T, torch, sbc, _lib, dev)
    if w["kind"] == "stream":
        return stream_main(a, w, T, torch, sbc, _lib, dev)
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

        # an uncapped search needs a capacity to run unsynchronised
        cap_ball = None if w["k_cap"] > 0 else sbc.neighbour_search_points(
            x_in, s_in, x_out, s_out, w["radius"], 0).nnz

        def search():
            return sbc.neighbour_search_points(x_in, s_in, x_out, s_out, w["radius"],
                                               w["k_cap"], col_capacity=cap_ball, sync=False)

        # the batch is block-diagonal: cloud by cloud, while a cloud's row
        # bounds fit the batched kernel's LDS (2048 rows); larger clouds take
        # the general transpose
        by_cloud = int(np.diff(w["out_splits"]).max()) < 2048

        def transpose(csr):
            return (sbc.csr_transpose_batched(csr, s_out, s_in) if by_cloud
                    else sbc.csr_transpose(csr))
    else:
        px, py, tt = T(w["px"]), T(w["py"]), T(w["t"])
        if w["basis"] == "event_decays":
            geo = sbc.Geometry("event_decays", px=px, py=py, t=tt, decays=T(w["decays"]))
        else:
            geo = sbc.Geometry("event8", tau=w["tau"], px=px, py=py, t=tt)
        cap = sbc.neighbour_search_events(px, py, tt, w["width"], w["height"], w["window"]).nnz
        found = {}

        def search():  # the pattern and its transpose from one set of pixel lists
            csr, found["csc"] = sbc.neighbour_search_events_csc(
                px, py, tt, w["width"], w["height"], w["window"], col_capacity=cap, sync=False)
            return csr

        def transpose(csr):
            return found["csc"]

    n_in, n_out = w["n_in"], w["n_out"]
    csr0 = search()
    torch.cuda.synchronize()
    E = int(csr0.row_ptr[-1].item())
    plan = sbc.conv_plan(n_out, n_in, csr0.nnz, M, ci, co, F.dtype, a.order)

    if w.get("sampling"):
        # down-sampling for the next layer: the uncapped ball, then the sampler
        smp = w["sampling"]
        n_batch = len(w["in_splits"]) - 1
        max_cloud = int(np.diff(w["in_splits"]).max())

        def step():
            csr = search()
            return sbc.sample_points(x_in, s_in, smp["method"], smp["per_cloud"], ball=csr,
                                     max_cloud=max_cloud)

        table = sampling_table(n_in, E, n_batch)
    elif w.get("featureless"):
        # the first layer on bare coordinates: Phi_0 = W[:, 0, :], dZ = dY
        Phi = W[:, 0, :].contiguous()

        def step():
            csr = search()
            Z = sbc.featureless_forward(csr, Phi, geometry=geo)
            dPhi = sbc.featureless_backward(csr, dY, M, geometry=geo)
            return Z, dPhi

        table = featureless_table(n_in, n_out, E, M, co)
    else:
        decays = w["basis"] == "event_decays"

        in_step = w.get("search_in_step", True)

        def step():
            csr = search() if in_step else csr0
            Y = sbc.conv_forward(csr, F, W, geometry=geo, order=a.order)
            csc = transpose(csr)
            dF, dW = sbc.conv_backward(csr, csc, F, W, dY, geometry=geo, order=a.order)
            if decays:  # the learned decay rates are parameters too
                return Y, dF, dW, sbc.conv_decay_gradient(csr, F, W, dY, geo, csc=csc)
            return Y, dF, dW

        n_cus = torch.cuda.get_device_properties(dev).multi_processor_count
        tr_bwd = 32                                       # the fused backward's tile rows
        blocks_bwd = max(1, min(256, n_cus, (n_in + tr_bwd - 1) // tr_bwd))
        npix = w["width"] * w["height"] if w["kind"] == "events" else 0
        table = kernel_table(w["kind"], plan, n_in, n_out, E, M, ci, co, sf, blocks_bwd, npix)
        if not in_step:
            for k in ("points_count", "points_fill"):
                table.pop(k, None)
        if w["kind"] == "points" and not by_cloud:
            # the general transpose: column counts, a scatter, then the
            # in-column ordering
            table.pop("transpose_batched")
            table["transpose_count"] = (1, 4 * (n_out + 1) + 4 * E + 4 * n_in, 0, False)
            table["transpose_scatter"] = (1, 4 * (n_out + 1) + 4 * E + 12 * E, 0, False)
            table["transpose_sort"] = (1, 4 * (n_in + 1) + 16 * E, 0, False)
        if decays:
            if plan["backward_fused"]:
                # the fused D-route with the derivative values, dF skipped
                table["decay_fused"] = (1, 4 * (n_in + 1) + 4 * E + 12 * n_in + n_out * co * sf
                                        + n_in * ci * sf, 2 * n_in * M * ci * co, True)
                table["decay_dw_reduce"] = (1, 4 * M * ci * co, 0, False)
            else:
                G_b = 4 * n_out * M * ci
                table["decay_basis"] = (1, 4 * (n_out + 1) + 4 * E + 12 * n_in + 4 * E * M, 0,
                                        False)
                table["decay_spmm"] = (1, 4 * (n_out + 1) + 8 * E + 4 * E * M + n_in * ci * sf
                                       + G_b, 2 * E * M * ci, False)
                table["decay_gemm"] = (1, G_b + n_out * co * sf + 4 * M * ci * co,
                                       2 * n_out * M * ci * co, True)
            table["decay_dot"] = (1, 4 * M * ci * co + M * ci * co * sf + 4 * M, 0, False)
    ms, eager_ms, wall, kernels, roof, dist = measure(a, w, table, step, torch, _lib, dev)
    dt = w["dtype"]
    # the paper's own number for this exact workload: Table 2's full training
    # pass (4.1 ms, N(F Theta) with JIT) over the same 294,912 edges, on a
    # GTX-1080Ti; the search is left out on both sides
    vs = E / (ms * 1e-3) / (E / 4.1e-3) if a.workload == "table2_flexconv" else None
    out = {"metric": METRIC, "value": E / (ms * 1e-3), "unit": "edges/s", "n_gpus": 1,
           "steps": a.steps, "warmup": a.warmup, "ms_per_step": round(ms, 4),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": vs, "dtype": dt,
           "data": "synthetic (seeded generators; inputs resident in HBM)",
           "config": {"workload": f"{a.workload}: {DESCRIPTIONS[a.workload]}", "n_in": n_in,
                      "n_out": n_out, "edges": E, "M": M, "C_in": ci, "C_out": co,
                      "plan": plan,
                      "timing": "eager steps" if a.no_graph else "HIP graph replays of the captured step",
                      "eager_ms_per_step": round(eager_ms, 4), "wall_s": round(wall, 3),
                      "replays": dist},
           "roofline": roof, "kernels": kernels}
    if not a.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, a.cpu_reps)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
