"""Host-side checks of bench.py: the one-GPU rule and the traffic record
lookup (no GPU needed)."""
import glob
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402

RECORDS = sorted(glob.glob(os.path.join(ROOT, "profiles", "extract_*_traffic.json")))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_the_benchmark_workload_has_a_traffic_record():
    assert os.path.join(ROOT, "profiles", "extract_qwen3_8b_tp4_traffic.json") in RECORDS


@pytest.mark.parametrize("path", RECORDS, ids=[os.path.basename(p) for p in RECORDS])
def test_traffic_record_lookup(path):
    from paper_2608_00455_amd import devcode
    rec = json.load(open(path))
    workload = os.path.basename(path)[len("extract_"):-len("_traffic.json")]
    got = bench.measured_traffic(workload, "extract", rec["mode"])
    lib = os.path.join(ROOT, rec["library"])
    if not os.path.exists(lib) or \
            devcode.kernel_sha256(lib, rec["kernel_symbols"]) != rec["device_code_sha256"]:
        # the built kernels are not the ones the counters were taken on
        assert got is None
        return
    assert got == rec["traffic_bytes_per_launch"]
    # the fetch and write counters, scaled by the copy calibration, give the total
    cal = rec["copy_calibration"]
    total = (sum(rec["fetch_size_kib_per_call"].values()) * 1024 * cal["fetch_factor"] +
             sum(rec["write_size_kib_per_call"].values()) * 1024 * cal["write_factor"])
    assert abs(total - got) < 1.0
    # within about one percent of extract's algorithmic bytes 12 N + 10 M
    # (the dense sweep point writes partial lines at the ends of its runs:
    # its WRITE_SIZE is about 1.1 x its 10 M bytes)
    assert 1.0 <= got / rec["algorithmic_bytes_per_launch"] < 1.02


def test_traffic_is_withheld_for_another_mode_or_workload():
    assert bench.measured_traffic("qwen3_8b_tp4", "extract", "no such mode") is None
    assert bench.measured_traffic("no_such_workload", "extract", "unordered") is None


APPLY_RECORDS = sorted(glob.glob(os.path.join(ROOT, "profiles", "apply_*_traffic.json")))


@pytest.mark.parametrize("path", APPLY_RECORDS, ids=[os.path.basename(p) for p in APPLY_RECORDS])
def test_apply_traffic_record_lookup(path):
    """Apply-only records: the lookup returns the recorded bytes while the
    built apply kernel is the profiled one; scattered 2-byte stores cost
    whole sectors, so the bytes exceed the algorithmic ones."""
    from paper_2608_00455_amd import devcode
    rec = json.load(open(path))
    workload = os.path.basename(path)[len("apply_"):-len("_traffic.json")]
    got = bench.measured_traffic(workload, "apply", rec["mode"])
    lib = os.path.join(ROOT, rec["library"])
    if not os.path.exists(lib) or \
            devcode.kernel_sha256(lib, rec["kernel_symbols"]) != rec["device_code_sha256"]:
        assert got is None
        return
    assert got == rec["traffic_bytes_per_launch"]
    assert got > rec["algorithmic_bytes_per_launch"]
