"""Summaries of rocprofv3 output for the benchmark's records.

  kernel_stats(csv)            per-kernel calls and durations of a
                               `rocprofv3 --kernel-trace --stats` run
  pmc_per_dispatch(csv, sub)   mean counter value per dispatch of every
                               kernel whose name contains `sub`, from a
                               `rocprofv3 --pmc <counter>` run
  traffic_record(...)          HBM bytes per call of a kernel family from
                               one FETCH_SIZE and one WRITE_SIZE run, each
                               scaled by what the same counter reads for a
                               plain device copy of known size, tied to the
                               built kernels' machine code

    python -m paper_2608_00455_amd.profiling stats <kernel_stats.csv>
    python -m paper_2608_00455_amd.profiling traffic --kernel extract_kernel \\
        --fetch F.csv --write W.csv --copy-fetch CF.csv --copy-write CW.csv \\
        --copy-bytes 4294967296 --algorithmic-bytes B --mode unordered \\
        --workload NAME --note TEXT --out profiles/extract_NAME_traffic.json
"""
from __future__ import annotations

import argparse
import csv
import json
import os
import sys
from collections import OrderedDict

from . import devcode

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB_REL = os.path.relpath(os.path.join(HERE, "libdte.so"), ROOT)


def kernel_stats(path):
    """[(name, calls, average_ms, min_ms, max_ms)] in the file's order."""
    out = []
    with open(path, newline="") as f:
        for row in csv.DictReader(f):
            out.append((row["Name"], int(row["Calls"]), float(row["AverageNs"]) / 1e6,
                        float(row["MinNs"]) / 1e6, float(row["MaxNs"]) / 1e6))
    return out


def pmc_per_dispatch(path, name_substring):
    """{kernel name: (dispatches, mean counter value)} over the dispatches
    of kernels whose name contains name_substring (one counter per file)."""
    acc = OrderedDict()
    counter = None
    with open(path, newline="") as f:
        for row in csv.DictReader(f):
            if name_substring not in row["Kernel_Name"]:
                continue
            if counter is None:
                counter = row["Counter_Name"]
            elif row["Counter_Name"] != counter:
                raise ValueError("%s holds more than one counter" % path)
            n, s = acc.get(row["Kernel_Name"], (0, 0.0))
            acc[row["Kernel_Name"]] = (n + 1, s + float(row["Counter_Value"]))
    return OrderedDict((k, (n, s / n)) for k, (n, s) in acc.items())


def _copy_factor(path, nbytes):
    per = pmc_per_dispatch(path, "copyBuffer")
    if not per:
        raise ValueError("no copy kernel in %s" % path)
    kib = max(v for _, v in per.values())
    return kib, nbytes / (kib * 1024.0)


def traffic_record(kernel, fetch, write, copy_fetch, copy_write, copy_bytes, algorithmic_bytes,
                   mode, workload, note=""):
    f = pmc_per_dispatch(fetch, kernel)
    w = pmc_per_dispatch(write, kernel)
    cf_kib, cf = _copy_factor(copy_fetch, copy_bytes)
    cw_kib, cw = _copy_factor(copy_write, copy_bytes)
    traffic = (sum(v for _, v in f.values()) * 1024.0 * cf +
               sum(v for _, v in w.values()) * 1024.0 * cw)
    return OrderedDict([
        ("kernel_symbols", kernel),
        ("library", LIB_REL),
        ("device_code_sha256", devcode.kernel_sha256(os.path.join(ROOT, LIB_REL), kernel)),
        ("mode", mode),
        ("workload", workload),
        ("fetch_size_kib_per_call", OrderedDict((k, v) for k, (_, v) in f.items())),
        ("write_size_kib_per_call", OrderedDict((k, v) for k, (_, v) in w.items())),
        ("dispatches_averaged", OrderedDict((k, n) for k, (n, _) in f.items())),
        ("copy_calibration", OrderedDict([("bytes_read", copy_bytes), ("fetch_size_kib", cf_kib),
                                          ("fetch_factor", cf), ("bytes_written", copy_bytes),
                                          ("write_size_kib", cw_kib), ("write_factor", cw)])),
        ("traffic_bytes_per_launch", traffic),
        ("algorithmic_bytes_per_launch", algorithmic_bytes),
        ("traffic_over_algorithmic", traffic / algorithmic_bytes if algorithmic_bytes else None),
        ("note", note),
    ])


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("csv")
    t = sub.add_parser("traffic")
    for a in ("kernel", "fetch", "write", "copy-fetch", "copy-write", "mode", "workload", "out"):
        t.add_argument("--" + a, required=True)
    t.add_argument("--copy-bytes", type=int, required=True)
    t.add_argument("--algorithmic-bytes", type=int, required=True)
    t.add_argument("--note", default="")
    a = ap.parse_args(argv)
    if a.cmd == "stats":
        print("| kernel | calls | average ms | min ms | max ms |")
        print("|---|---|---|---|---|")
        for name, calls, avg, mn, mx in kernel_stats(a.csv):
            print("| %s | %d | %.4f | %.4f | %.4f |" % (name, calls, avg, mn, mx))
        return 0
    rec = traffic_record(a.kernel, a.fetch, a.write, a.copy_fetch, a.copy_write, a.copy_bytes,
                         a.algorithmic_bytes, a.mode, a.workload, a.note)
    with open(a.out, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec))
    return 0


if __name__ == "__main__":
    sys.exit(main())
