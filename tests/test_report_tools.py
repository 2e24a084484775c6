"""Host-side tools behind the benchmark's records: the oracle's CPU timing
(oracle/timing.py), the rocprofv3 CSV summaries (profiling.py) and the
fingerprint of the built kernels (devcode.py)."""
import csv
import os

import pytest

from oracle import run as orun
from oracle import timing
from paper_2608_00455_amd import build as dte_build
from paper_2608_00455_amd import devcode, profiling
from synth import workloads as W


def test_oracle_timing_runs_both_ways_and_counts_the_delta():
    wl = W.scaled_dense(layers=1, tp=2, lr=1e-5)
    r = timing.time_workload(wl, procs=2, reps=1, window=1 << 15, gen_threads=2)
    assert r["changed"] == orun.extract(wl, threads=2).idx.size > 0
    assert r["elements"] == wl.numel and r["procs"] == 2 and r["windows"] > 2
    assert r["single_process_s"] > 0 and r["pool_s"] > 0
    assert r["pool_elements_per_s"] == pytest.approx(wl.numel / r["pool_s"])
    assert timing.workload("qwen3_8b_4l_tp4_lr1e-05").hp.lr == 1e-5
    with pytest.raises(ValueError):
        timing.workload("no_such_workload")
    assert timing.cpu_model()


def _write(path, header, rows):
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)
    return str(path)


def test_profiling_summaries(tmp_path):
    ks = _write(tmp_path / "ks.csv", ["Name", "Calls", "AverageNs", "MinNs", "MaxNs"],
                [["extract_kernel", 3, 2_000_000, 1_500_000, 2_500_000]])
    assert profiling.kernel_stats(ks) == [("extract_kernel", 3, 2.0, 1.5, 2.5)]
    H = ["Kernel_Name", "Counter_Name", "Counter_Value"]
    fetch = _write(tmp_path / "f.csv", H, [["extract_kernel<a>", "FETCH_SIZE", 100.0],
                                          ["extract_kernel<a>", "FETCH_SIZE", 300.0],
                                          ["extract_kernel<b>", "FETCH_SIZE", 8.0],
                                          ["remap_kernel", "FETCH_SIZE", 5.0]])
    write = _write(tmp_path / "w.csv", H, [["extract_kernel<a>", "WRITE_SIZE", 50.0],
                                          ["extract_kernel<a>", "WRITE_SIZE", 50.0]])
    per = profiling.pmc_per_dispatch(fetch, "extract_kernel")
    assert per == {"extract_kernel<a>": (2, 200.0), "extract_kernel<b>": (1, 8.0)}
    mixed = _write(tmp_path / "x.csv", H, [["k", "FETCH_SIZE", 1], ["k", "WRITE_SIZE", 1]])
    with pytest.raises(ValueError):
        profiling.pmc_per_dispatch(mixed, "k")
    # a 4 KiB copy that reads as 2 KiB of FETCH_SIZE and 4 KiB of WRITE_SIZE
    cf = _write(tmp_path / "cf.csv", H, [["__amd_rocclr_copyBuffer", "FETCH_SIZE", 2.0]])
    cw = _write(tmp_path / "cw.csv", H, [["__amd_rocclr_copyBuffer", "WRITE_SIZE", 4.0]])
    if not os.path.exists(dte_build.LIB):
        pytest.skip("libdte.so not built")
    rec = profiling.traffic_record("extract_kernel", fetch, write, cf, cw, 4096, 1000, "unordered",
                                   "w", "n")
    assert rec["copy_calibration"]["fetch_factor"] == 2.0
    assert rec["copy_calibration"]["write_factor"] == 1.0
    assert rec["traffic_bytes_per_launch"] == (200.0 + 8.0) * 1024 * 2 + 50.0 * 1024
    assert rec["device_code_sha256"] == devcode.kernel_sha256(dte_build.LIB, "extract_kernel")


def test_device_code_fingerprint():
    if not os.path.exists(dte_build.LIB):
        pytest.skip("libdte.so not built")
    a = devcode.kernel_sha256(dte_build.LIB, "extract_kernel")
    assert len(a) == 64 and int(a, 16) >= 0
    assert a == devcode.kernel_sha256(dte_build.LIB, "extract_kernel")
    assert a != devcode.kernel_sha256(dte_build.LIB, "remap_kernel") != ""
    assert devcode.kernel_sha256(dte_build.LIB, "no_such_kernel") == ""
    assert devcode.kernel_sha256(dte_build.LIB, "extract_kernel", arch="gfx000") == ""
