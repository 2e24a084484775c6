#!/usr/bin/env python3
"""Throughput of the delta-extraction hot path on one MI355X.

One step = one pass of the whole path over the trainer shard already
resident in HBM: reset the delta cursor, dte_extract_delta (AdamW
inversion + BF16 change detection + compaction; --ordered:
dte_extract_delta_ordered, an ascending delta), dte_remap (receiver
coordinates) and dte_apply (scatter into the receiver BF16 shards).

Default workload: the full Qwen3-8B state (8,190,735,360 fp32 elements of
theta, m, v; receiver TP=4).  Prints one JSON line with the throughput in
elements/s, the roofline of the dominant kernel (extract, HBM-bound) and
the CPU oracle's throughput on a bounded sample of the same workload.

Other workloads (--workload): tiny_block_tp2, qwen3_30b_a3b_12l_ep8,
qwen3_8b_4l_tp4 (with --lr), qwen3_8b_4l_mcore (four Qwen3-8B layers held as
the Megatron-Core shard of trainer TP rank 1 of 2, receiver TP=4),
qwen3_8b_tp8_apply (apply-only timing of the Qwen3-8B delta into eight TP=8
shards).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E peak


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def workload(name, lr):
    import synth
    from synth import workloads as W
    if name == "qwen3_8b_tp4":
        return W.qwen3_8b(4)
    if name == "qwen3_8b_tp8_apply":
        return W.qwen3_8b(8)
    if name == "tiny_block_tp2":
        return W.tiny_block()
    if name == "qwen3_30b_a3b_12l_ep8":
        return W.qwen3_30b_a3b_share(synth.word)
    if name == "qwen3_8b_4l_tp4":
        return W.qwen3_8b_layers_sweep(lr if lr is not None else 1e-6)
    if name == "qwen3_8b_4l_mcore":
        return W.qwen3_8b_layers_mcore(trainer_rank=1, lr=lr if lr is not None else 1e-6)
    raise SystemExit("unknown workload %r" % name)


def cpu_baseline(seconds_target=10.0):
    """The oracle (inversion, BF16 detection, nonzero, remap, apply) timed
    on the host cores over a bounded sample of the default workload: one
    Qwen3-8B layer (192,946,432 elements, receiver TP=4), its post-step
    state generated once untimed, then whole oracle passes over it repeated
    until at least `seconds_target` seconds of oracle work are timed."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import synth
    from oracle import core, plan, remap, run
    from synth import workloads as W

    threads = synth.default_threads()
    wl = W.qwen3_8b_layers_sweep(1e-6, layers=1)
    pl = plan.build_plan(wl)
    sc = core.derive_scalars(wl.hp)
    wins = run.windows(wl, 1 << 22)
    begins = wl.flat_begins()
    with ThreadPoolExecutor(threads) as ex:
        states = list(ex.map(lambda w: run.state(wl, w.tensor, w.lo, w.hi, sc), wins))
    shards = [np.zeros(n, np.uint16) for n in pl.rank_numel]

    def one_pass(ex):
        parts = list(ex.map(
            lambda a: core.detect(a[1][1], a[1][2], a[1][3], sc, begins[a[0].tensor] + a[0].lo)[:2],
            zip(wins, states)))
        idx = np.concatenate([x[0] for x in parts])
        val = np.concatenate([x[1] for x in parts])
        remap.apply(shards, remap.remap(pl, idx, val))

    secs, passes = 0.0, 0
    with ThreadPoolExecutor(threads) as ex:
        while secs < seconds_target and passes < 200:
            t0 = time.perf_counter()
            one_pass(ex)
            secs += time.perf_counter() - t0
            passes += 1
    return {"value": passes * wl.numel / secs, "unit": "elements/s", "cores": threads,
            "kind": "oracle",
            "sample": "%d passes over one Qwen3-8B layer (%d elements, receiver TP=4, "
                      "lr 1e-6): inversion + BF16 detection + nonzero + remap + apply, "
                      "%d threads; state generated once, untimed; %s"
                      % (passes, wl.numel, threads, run.host_description()),
            "seconds": secs}


def measured_traffic(workload_name, kernel, mode):
    """HBM bytes per call of the dominant kernel(s) from the committed
    rocprofv3 FETCH_SIZE / WRITE_SIZE record (scaled by a plain copy's
    counter reading), or None when there is no record for this workload and
    mode or the kernel source changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "%s_%s_traffic.json" % (kernel, workload_name))
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("mode") != mode:
        return None
    src = os.path.join(ROOT, rec["kernel_source"])
    if hashlib.sha256(open(src, "rb").read()).hexdigest() != rec["kernel_source_sha256"]:
        return None
    return rec["traffic_bytes_per_launch"]


def storage_leg(root, wl, spec, p, m, v, hp, cap):
    """Publish one ordered delta through the storage path (writer part +
    commit: device narrowing, pinned staging, zstd level 3 on 16 host
    threads, files, manifest) and read it back into device memory; host
    wall-clock times, not part of the step."""
    import shutil

    import torch

    from paper_2608_00455_amd import store as S
    from paper_2608_00455_amd.pipeline import DeltaPipeline

    d = os.path.join(root, "dte_store_bench")
    shutil.rmtree(d, ignore_errors=True)
    pipe = DeltaPipeline(spec, capacity=cap, ordered=True)
    pipe.reset()
    pipe.extract(p, m, v, hp)
    torch.cuda.synchronize()
    segs = S.segments_of([t.name for t in wl.tensors], wl.flat_begins(),
                         [t.numel for t in wl.tensors])
    opt = S.Options(threads=16)
    t0 = time.perf_counter()
    st = S.write_part_device(d, 1, 0, segs, pipe.idx.data_ptr(), pipe.val.data_ptr(),
                             pipe.cursor.data_ptr(), pipe.capacity, opt)
    S.commit(d, 1, 0, 1)
    t1 = time.perf_counter()
    n, _ = S.read_device(d, 1, 0, pipe.idx.data_ptr(), pipe.val.data_ptr(), pipe.capacity,
                         threads=16)
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    pipe.close()
    shutil.rmtree(d, ignore_errors=True)
    return {"entries": int(n), "chunks": st.chunks, "raw_bytes": st.raw_bytes,
            "stored_bytes": st.stored_bytes, "ratio": st.raw_bytes / max(1, st.stored_bytes),
            "publish_s": t1 - t0, "read_s": t2 - t1, "codec": "zstd-3", "threads": 16}


def copy_calibration(gib):
    """A plain copy of known size: reads and writes gib GiB once per launch."""
    import torch
    n = int(gib * (1 << 30)) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(2):
        dst.copy_(src)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    reps = 5
    for _ in range(reps):
        dst.copy_(src)
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    print(json.dumps({"copy_bytes_read": 4 * n, "copy_bytes_written": 4 * n, "ms": ms,
                      "gbs_read_plus_write": 8 * n / (ms / 1e3) / 1e9}), flush=True)
    return 0


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="qwen3_8b_tp4")
    ap.add_argument("--lr", type=float, default=None)
    ap.add_argument("--literal", action="store_true",
                    help="literal operation order of the AdamW inverse (four divisions)")
    ap.add_argument("--fused", action="store_true",
                    help="dte_extract_remap (detection routed straight into the buckets) "
                         "instead of dte_extract_delta + dte_remap")
    ap.add_argument("--ordered", action="store_true",
                    help="dte_extract_delta_ordered (ascending, deterministic delta)")
    ap.add_argument("--norm-group", action="store_true",
                    help="norms in a parameter group without weight decay")
    ap.add_argument("--capacity-fraction", type=float, default=None,
                    help="delta buffer size as a fraction of the elements (default 0.02, "
                         "0.25 for the learning-rate sweep)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--settle", type=float, default=15.0, metavar="SECONDS",
                    help="wait before allocating the state: device memory that a process "
                         "released moments earlier is handed out in less contiguous pieces "
                         "until the driver has reclaimed it, which slows streaming kernels")
    ap.add_argument("--store", default=None, metavar="DIR",
                    help="also publish the step's delta through the storage path (ordered "
                         "extract, zstd chunks under DIR) and read it back to the device; "
                         "reports the times and sizes under 'storage'")
    ap.add_argument("--copy-calibration", type=float, default=0.0, metavar="GIB",
                    help="only time a plain device copy of GIB GiB (for scaling the "
                         "FETCH_SIZE / WRITE_SIZE counters) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU; the multi-GPU exchange is not implemented "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr)
        return 2

    import torch

    from paper_2608_00455_amd import layouts
    from paper_2608_00455_amd.pipeline import DeltaPipeline, generate_state, group_runs
    from synth import workloads as W

    torch.cuda.set_device(0)
    if args.copy_calibration > 0:
        return copy_calibration(args.copy_calibration)
    wl = workload(args.workload, args.lr)
    if args.norm_group:
        wl = W.with_norm_group(wl)
    hp = wl.hp if args.lr is None else type(wl.hp)(lr=args.lr)
    if args.literal:
        hp = type(hp)(lr=hp.lr, beta1=hp.beta1, beta2=hp.beta2, eps=hp.eps,
                      weight_decay=hp.weight_decay, step=hp.step, order=W.ORDER_LITERAL)
    if args.settle > 0:
        log("bench: settling %.0f s before allocating" % args.settle)
        time.sleep(args.settle)
    spec = layouts.build_spec(wl)
    n = spec.total                           # elements of the trainer shard
    log("bench: workload %s, %d elements, lr %g" % (wl.name, n, hp.lr))
    t = time.perf_counter()
    p, m, v = generate_state(wl, hp)
    log("bench: state generated in %.1f s" % (time.perf_counter() - t))
    frac = args.capacity_fraction
    if frac is None:
        frac = 0.25 if args.workload == "qwen3_8b_4l_tp4" else 0.02
    cap = max(1 << 20, int(n * frac))
    ordered = bool(args.ordered)
    pipe = DeltaPipeline(spec, capacity=cap, ordered=ordered)
    runs = group_runs(wl, hp)
    stream = torch.cuda.current_stream()
    apply_only = args.workload.endswith("_apply")

    def step(ev=None):
        if apply_only:
            if ev:
                ev[0].record(stream)
            pipe.apply()
            if ev:
                ev[1].record(stream)
            return
        if args.fused:
            pipe.cursor.zero_()
            pipe.rank_count.zero_()
            if ev:
                ev[0].record(stream)
            for b, e, h in runs:
                if len(runs) == 1:
                    pipe.extract_remap(p, m, v, h)
                else:
                    pipe.extract_remap(p[b:e], m[b:e], v[b:e], h, n=e - b, index_base=b)
            if ev:
                ev[1].record(stream)
                ev[2].record(stream)
        else:
            pipe.reset()
            if ev:
                ev[0].record(stream)
            if len(runs) == 1:
                pipe.extract(p, m, v, hp)
            else:
                pipe.extract_runs(p, m, v, runs)
            if ev:
                ev[1].record(stream)
            pipe.remap()
            if ev:
                ev[2].record(stream)
        pipe.apply()
        if ev:
            ev[3].record(stream)

    if apply_only:                           # delta and buckets prepared untimed
        pipe.step(p, m, v, hp)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    nev = 2 if apply_only else 4
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(nev)] for _ in range(args.steps)]
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for k in range(args.steps):
        step(evs[k])
    end.record(stream)
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    ms_step = total_ms / args.steps
    changed = int(pipe.cursor.item())
    counts = pipe.rank_count.cpu().tolist()
    routed = int(sum(counts))
    if changed > cap or any(c > cap for c in counts):
        log("bench: capacity exceeded (changed %d, capacity %d)" % (changed, cap))
        return 3
    c = changed / n

    if apply_only:
        k_ms = sum(e[0].elapsed_time(e[1]) for e in evs) / args.steps
        k_bytes = routed * (8 + 2 + 2)       # read offset + value, write value
        value = routed / (ms_step / 1e3)
        metric_unit = "entries/s"
        kernel = "apply"
    else:
        ext_ms = sum(e[0].elapsed_time(e[1]) for e in evs) / args.steps
        rem_ms = sum(e[1].elapsed_time(e[2]) for e in evs) / args.steps
        app_ms = sum(e[2].elapsed_time(e[3]) for e in evs) / args.steps
        k_ms = ext_ms
        if args.fused:                        # read theta, m, v; write (offset, value) per route
            k_bytes = 12 * n + 10 * routed
        else:                                 # read theta, m, v; write (idx, val)
            k_bytes = 12 * n + 10 * changed
        value = n / (ms_step / 1e3)
        metric_unit = "elements/s"
        kernel = "extract_remap" if args.fused else "extract"
    if apply_only:
        step_bytes = k_bytes
    elif args.fused:
        step_bytes = 12 * n + 10 * routed + 12 * routed
    else:
        step_bytes = 12 * n + 10 * changed + 10 * changed + 10 * routed + 12 * routed
    achieved = k_bytes / (k_ms / 1e3) / 1e9
    # the counters were taken for the default configuration only (folded
    # order, unordered output, one parameter group)
    default_mode = not (args.ordered or args.fused or args.literal or args.norm_group)
    out = {
        "metric": "delta-extract+remap+apply: elements/s and HBM GB/s (% of peak), "
                  "Qwen3-8B shape",
        "value": value,
        "unit": metric_unit,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded Philox draws, one AdamW step on the device)",
        "config": {"workload": wl.name, "elements": n, "changed": changed, "extract_calls": len(runs), "settle_s": args.settle,
                   "ordered": ordered, "fused": bool(args.fused), "order": "literal" if args.literal else "folded",
                   "change_fraction": c, "receiver_ranks": len(counts),
                   "routed_entries": routed, "lr": hp.lr,
                   "step_algorithmic_bytes": step_bytes,
                   "step_gbs": step_bytes / (ms_step / 1e3) / 1e9,
                   "step_frac_of_hbm_peak": step_bytes / (ms_step / 1e3) / 1e9 / HBM_PEAK_GBS},
        "roofline": {"kernel": kernel, "bound": "hbm", "achieved": achieved,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": (measured_traffic(wl.name, kernel, "unordered")
                                 if default_mode else None),
                     "kernel_ms": k_ms,
                     "bytes_per_launch": k_bytes},
    }
    if not apply_only:
        out["config"].update({"extract_ms": ext_ms, "remap_ms": rem_ms, "apply_ms": app_ms})
    if args.store and not apply_only:
        out["storage"] = storage_leg(args.store, wl, spec, p, m, v, hp, cap)
    del p, m, v
    pipe.close()
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        log("bench: timing the CPU oracle on a sample")
        out["cpu_baseline"] = cpu_baseline(args.cpu_seconds)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
