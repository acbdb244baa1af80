"""Host logic of bench.py that needs no GPU: the one-GPU guard, the mapping of
profiled kernels to the library's trace names, the traffic summary with its
copy-probe calibration and source fingerprints, and the workloads' shapes."""
import csv
import json
import os
import subprocess
import sys

import numpy as np
import pytest

import bench
import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


@pytest.mark.parametrize("kernel,name", [
    ("bwd_ws_kernel<8, 64, 64, 2, false, 4, 4, 32, 0>", "bwd_fused"),
    ("bwd_ws_kernel<16, 32, 32, 16, false, 4, 4, 32, 0>", "decay_fused"),
    ("fwd_reg_kernel<8, 32, 32, 3, false>", "fwd_fused"),
    ("fwd_onehot_kernel<32, 32>", "fwd_fused"),
    ("featureless_kernel<10, 3, true>", "featureless_fwd"),
    ("featureless_kernel<10, 3, false>", "featureless_rowsum"),
    ("sample_kernel<true>", "sample"),
    ("sample_kernel<false>", "sample_count"),
    ("lif_cell_kernel<3>", "lif_cells"),
    ("gemm_kernel<64, 64, float, float, true, true>", None),
    ("spmm_kernel<8, true, float>", "spmm_contract"),
    ("spmm_kernel<10, false, unsigned short>", "spmm_expand"),
])
def test_trace_names(kernel, name):
    assert bench.trace_name(kernel) == name


def test_spmm_launches_file_their_counters_by_direction():
    """Every launch of the generic gather maps onto the counter line of its
    direction, so a workload's dominant gather finds its measured bytes."""
    assert bench.SPMM_DIRECTION["bwd_spmm_t"] == "spmm_contract"
    assert bench.SPMM_DIRECTION["fwd_spmm_contract"] == "spmm_contract"
    for n in ("fwd_spmm", "bwd_spmm", "bwd_spmm_t_expand", "decay_spmm"):
        assert bench.SPMM_DIRECTION[n] == "spmm_expand"


def _counter_dir(tmp_path, tag, counter, rows):
    d = tmp_path / tag
    d.mkdir()
    with open(d / "p_counter_collection.csv", "w", newline="") as f:
        wr = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value"])
        wr.writeheader()
        for k, v in rows:
            wr.writerow({"Kernel_Name": k, "Counter_Name": counter, "Counter_Value": v})
    return str(d)


def test_traffic_summary_is_calibrated_by_the_copy_probe(tmp_path):
    """A 1 MiB probe whose FETCH_SIZE reads 512 KiB gives a fetch factor of 2;
    a kernel reading 100 KiB and writing 50 KiB per dispatch then moves
    (200 + 50) KiB, and its line carries the fingerprint of its source."""
    k = "void sbc::(anonymous namespace)::bwd_ws_kernel<8, 64, 64, 2, false, 4, 4, 32, 0>(A)"
    fetch = _counter_dir(tmp_path, "fetch", "FETCH_SIZE",
                         [("__amd_rocclr_copyBuffer", 512.0), (k, 100.0), (k, 100.0)])
    write = _counter_dir(tmp_path, "write", "WRITE_SIZE",
                         [("__amd_rocclr_copyBuffer", 1024.0), (k, 50.0), (k, 50.0)])
    text = bench.summarize_traffic(fetch, write, 1, "cmd")
    line = [l for l in text.splitlines() if l.startswith("traffic bwd_fused")][0].split()
    assert float(line[5]) == pytest.approx(250 * 1024)
    assert line[6] == bench.kernel_fingerprint("bwd_ws_kernel")


def test_counter_summary_averages_dispatches_and_drops_small_kernels(tmp_path):
    """Per kernel, a counter's readings are averaged over dispatches; kernels
    under 2% of the largest one's wave-cycles are left out."""
    big = "void sbc::(anonymous namespace)::fwd_reg_kernel<8, 32, 32, 3, false>(A)"
    small = "void sbc::(anonymous namespace)::pack_events_kernel(A)"
    d = tmp_path / "sq"
    d.mkdir()
    with open(d / "a_counter_collection.csv", "w", newline="") as f:
        wr = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name",
                                           "Counter_Value"])
        wr.writeheader()
        for i, v in ((1, 100.0), (2, 300.0)):
            wr.writerow({"Dispatch_Id": i, "Kernel_Name": big, "Counter_Name": "SQ_WAVE_CYCLES",
                         "Counter_Value": v})
            wr.writerow({"Dispatch_Id": i, "Kernel_Name": big, "Counter_Name": "SQ_INSTS_VALU",
                         "Counter_Value": 2 * v})
        wr.writerow({"Dispatch_Id": 3, "Kernel_Name": small, "Counter_Name": "SQ_WAVE_CYCLES",
                     "Counter_Value": 1.0})
    text = bench.summarize_counters([str(d)], "cmd")
    assert "kernel fwd_reg_kernel<8, 32, 32, 3, false>" in text
    assert "pack_events_kernel" not in text
    assert "SQ_WAVE_CYCLES 200  (2 dispatches)" in text
    assert "SQ_INSTS_VALU 400  (2 dispatches)" in text


def test_workload_shapes():
    """The benchmark workloads have the sizes their descriptions give."""
    w = workloads.table2_flexconv()
    assert w["n_in"] == w["n_out"] == 8 * 4096 and w["M"] == 4 and w["k_cap"] == 9
    assert w["C_in"] == w["C_out"] == 64 and not w["search_in_step"]
    w = workloads.events_300k_lif()
    assert w["n_in"] == 300_000 and (w["kernel"], w["stride"]) == (3, 2)
    assert np.all(np.diff(w["t"]) >= 0)
    w = workloads.events_stream()
    assert w["batch"] == 4096 and w["W"].shape == (8, 32, 32)
    assert set(workloads.WORKLOADS) <= set(bench.DESCRIPTIONS)
