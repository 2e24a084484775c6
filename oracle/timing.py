"""Host-core timing of the oracle -- TEST INFRASTRUCTURE ONLY (the
benchmark's CPU-baseline leg; the product path never imports it).

Times the method's steps after state generation: AdamW inversion
(sec. 4.1), BF16 detection and nonzero (sec. 4.2.1), receiver remap
(sec. 4.2.2) and direct apply (sec. 4.3) over a whole workload whose
post-step state was generated beforehand (untimed) and is held in host
memory, window by window (the oracle's per-tensor streaming):
  (i)  one process, one thread;
  (ii) a pool of P forked worker processes over the windows, each worker
       detecting and remapping its windows; the parent applies the buckets.
Both runs must produce the same receiver shards.

    python -m oracle.timing [--procs P] [--workloads tiny_block_tp2,qwen3_8b_4l_tp4_lr1e-06]
"""
from __future__ import annotations

import argparse
import json
import multiprocessing as mp
import os
import subprocess
import sys
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from synth import workloads as W

from . import core, plan, remap, run

_STATE = None     # inherited by the forked workers: (windows, states, plan, scalars, begins)


def cpu_model() -> str:
    """The `lscpu` model name (else /proc/cpuinfo's)."""
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=20).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    return run.host_description().split(",")[0]


def default_procs() -> int:
    return len(os.sched_getaffinity(0))


def _detect_remap(i):
    wins, states, pl, sc, begins = _STATE
    w = wins[i]
    p, m, v = states[i]
    idx, val, _ = core.detect(p, m, v, sc[w.tensor], begins[w.tensor] + w.lo)
    return idx.size, remap.remap(pl, idx, val)


def _apply_all(pl, results):
    shards = [np.zeros(n, np.uint16) for n in pl.rank_numel]
    changed = 0
    for cnt, buckets in results:
        changed += cnt
        remap.apply(shards, buckets)
    return changed, shards


def workload(name):
    if name == "tiny_block_tp2":
        return W.tiny_block()
    if name.startswith("qwen3_8b_4l_tp4_lr"):
        return W.qwen3_8b_layers_sweep(float(name[len("qwen3_8b_4l_tp4_lr"):]))
    raise ValueError("unknown workload %r" % name)


def time_workload(wl, procs: int, reps: int = 1, window: int = 1 << 22, gen_threads: int = 0):
    """Seconds of (i) one process and (ii) `procs` processes for inversion +
    detection + nonzero + remap + apply over all of `wl` (median of `reps`
    passes each); the post-step state is generated first, untimed."""
    global _STATE
    sc = run.scalars(wl)
    wins = run.windows(wl, window)
    begins = wl.flat_begins()
    gen_threads = gen_threads or min(16, procs)
    t0 = time.perf_counter()
    with ThreadPoolExecutor(gen_threads) as ex:
        states = list(ex.map(lambda w: run.state(wl, w.tensor, w.lo, w.hi, sc[w.tensor])[1:],
                             wins))
    pl = plan.build_plan(wl)
    gen_s = time.perf_counter() - t0
    _STATE = (wins, states, pl, sc, begins)
    try:
        single = []
        for _ in range(reps):
            t = time.perf_counter()
            changed, shards1 = _apply_all(pl, [_detect_remap(i) for i in range(len(wins))])
            single.append(time.perf_counter() - t)
        pooled = []
        with mp.get_context("fork").Pool(procs) as pool:
            pool.map(_detect_remap, [], chunksize=1)           # workers started, untimed
            for _ in range(reps):
                t = time.perf_counter()
                changed2, shards2 = _apply_all(pl, pool.map(_detect_remap, range(len(wins)),
                                                            chunksize=1))
                pooled.append(time.perf_counter() - t)
    finally:
        _STATE = None
    assert changed == changed2 and all(np.array_equal(a, b) for a, b in zip(shards1, shards2))
    single_s, pool_s = float(np.median(single)), float(np.median(pooled))
    return {"workload": wl.name, "elements": wl.numel, "changed": int(changed),
            "windows": len(wins), "reps": reps, "procs": procs,
            "single_process_s": single_s, "pool_s": pool_s,
            "single_process_elements_per_s": wl.numel / single_s,
            "pool_elements_per_s": wl.numel / pool_s, "generation_s_untimed": gen_s}


def baseline(procs: int = 0, names=("tiny_block_tp2", "qwen3_8b_4l_tp4_lr1e-06")) -> dict:
    procs = procs or default_procs()
    runs = []
    for name in names:
        wl = workload(name)
        reps = 5 if wl.numel < (1 << 26) else 1
        runs.append(time_workload(wl, procs, reps=reps))
    return {"procs": procs, "cpu_model": cpu_model(), "runs": runs}


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--procs", type=int, default=0)
    ap.add_argument("--workloads", default="tiny_block_tp2,qwen3_8b_4l_tp4_lr1e-06")
    a = ap.parse_args(argv)
    print(json.dumps(baseline(a.procs, tuple(a.workloads.split(",")))), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
