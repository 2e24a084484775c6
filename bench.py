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


def cpu_baseline(procs=0):
    """The oracle timed on the host cores: inversion, BF16 detection,
    nonzero, remap and apply over the tiny block and four Qwen3-8B layers at
    lr 1e-6 (a bounded sample of the benchmark's workload), their post-step
    states generated first (untimed); (i) in one process and (ii) with a
    pool of P processes.  `value` is the pool's rate on the four layers."""
    from oracle import timing

    res = timing.baseline(procs)
    big = res["runs"][-1]
    return {"value": big["pool_elements_per_s"], "unit": "elements/s", "cores": res["procs"],
            "kind": "oracle",
            "sample": "oracle inversion + BF16 detection + nonzero + remap + apply over every "
                      "element of %s; one process %.2f s, %d processes %.2f s; also %s; "
                      "states generated beforehand, untimed; %s"
                      % (big["workload"], big["single_process_s"], res["procs"], big["pool_s"],
                         ", ".join("%s %.3f / %.3f s" % (r["workload"], r["single_process_s"],
                                                         r["pool_s"])
                                   for r in res["runs"][:-1]), res["cpu_model"]),
            "cpu_model": res["cpu_model"], "procs": res["procs"],
            "single_process_elements_per_s": big["single_process_elements_per_s"],
            "runs": res["runs"]}


def measured_traffic(workload_name, kernel, mode):
    """HBM bytes per call of the dominant kernel(s) from the committed
    rocprofv3 FETCH_SIZE / WRITE_SIZE record (scaled by a plain copy's
    counter reading), or None when there is no record for this workload and
    mode or the built kernels' machine code differs from the code the
    counters were taken on."""
    from paper_2608_00455_amd import devcode
    path = os.path.join(ROOT, "profiles", "%s_%s_traffic.json" % (kernel, workload_name))
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("mode") != mode:
        return None
    lib = os.path.join(ROOT, rec["library"])
    if devcode.kernel_sha256(lib, rec["kernel_symbols"]) != rec["device_code_sha256"]:
        return None
    return rec["traffic_bytes_per_launch"]


def ceilings(p, m, v, pipe, stream, entries, reps=5, touch=None):
    """Second denominators measured on the same GPU and buffers: the rate of
    a plain read of theta, m, v (12 bytes per element, extract's access
    pattern, no arithmetic, no stores; best of 2, 3 and 4 blocks per CU
    with a static split and of one 12-wave block per CU taking four tiles
    per wave at a time);
    the writes of an `entries`-entry delta alone (8-byte offsets and 2-byte
    values spread evenly over the tiles, into the pipeline's delta buffers,
    which the step has finished with; same block counts), whose time added
    to the read's bounds any kernel that moves extract's bytes, and the
    same writes issued together with the read (a naive mix); and the time of
    writing whole 64-byte lines at every apply address of the step's
    buckets (into scratch buffers of the shards' size; best of 4, 8 and 16
    blocks per CU).  touch: run before every repetition, outside its
    events (the cache flush of a state that fits the last-level cache)."""
    import ctypes

    import torch

    from paper_2608_00455_amd import build as dte_build

    lib = ctypes.CDLL(dte_build.CEIL_LIB)
    P, I64, I32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    lib.ceil_read3_waves.restype = I64
    lib.ceil_read3_waves.argtypes = [I32]
    lib.ceil_read3.restype = ctypes.c_int
    lib.ceil_read3.argtypes = [P, P, P, I64, I32, P, P]
    lib.ceil_read3_dynamic.restype = ctypes.c_int
    lib.ceil_read3_dynamic.argtypes = [P, P, P, I64, P, P, P]
    lib.ceil_read3_write.restype = ctypes.c_int
    lib.ceil_read3_write.argtypes = [P, P, P, I64, I64, P, P, I32, P, P]
    lib.ceil_write_entries.restype = ctypes.c_int
    lib.ceil_write_entries.argtypes = [I64, P, P, I32, P]
    lib.ceil_line_writes.restype = ctypes.c_int
    lib.ceil_line_writes.argtypes = [I32, P, P, P, P, P, I32, P]
    s = stream.cuda_stream

    def timed(fn, name):
        best = None
        for _ in range(reps + 1):                       # the first is a warm-up
            if touch is not None:
                touch()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            rc = fn()
            if rc != 0:
                raise RuntimeError("%s failed (%d)" % (name, rc))
            b.record(stream)
            b.synchronize()
            ms = a.elapsed_time(b)
            best = ms if best is None or ms < best else best
        return best

    n = p.numel() // 2048 * 2048
    out = {}
    best = None
    for bpc in (2, 3, 4):
        sink = torch.zeros(64 * lib.ceil_read3_waves(bpc), dtype=torch.int32, device="cuda")
        ms = timed(lambda: lib.ceil_read3(p.data_ptr(), m.data_ptr(), v.data_ptr(), n, bpc,
                                          sink.data_ptr(), s), "ceil_read3")
        if best is None or ms < best[0]:
            best = (ms, "static", bpc, 4)
        del sink
    sink = torch.zeros(64 * lib.ceil_read3_waves(3), dtype=torch.int32, device="cuda")
    counter = torch.zeros(1, dtype=torch.int64, device="cuda")

    def dynamic_read():
        counter.zero_()
        return lib.ceil_read3_dynamic(p.data_ptr(), m.data_ptr(), v.data_ptr(), n,
                                      counter.data_ptr(), sink.data_ptr(), s)
    ms = timed(dynamic_read, "ceil_read3_dynamic")
    if ms < best[0]:
        best = (ms, "dynamic", 1, 12)
    del sink, counter
    out["read_stream"] = {"gbs": 12 * n / (best[0] / 1e3) / 1e9, "ms": best[0],
                          "split": best[1], "blocks_per_cu": best[2],
                          "waves_per_block": best[3], "bytes": 12 * n}
    e = min(entries, pipe.capacity)
    if e > 0:
        rd = best[0]
        wr = mix = None
        for bpc in (2, 3, 4):
            sink = torch.zeros(64 * lib.ceil_read3_waves(bpc), dtype=torch.int32, device="cuda")
            ms = timed(lambda: lib.ceil_write_entries(e, pipe.idx.data_ptr(), pipe.val.data_ptr(),
                                                      bpc, s), "ceil_write_entries")
            wr = ms if wr is None or ms < wr else wr
            ms = timed(lambda: lib.ceil_read3_write(p.data_ptr(), m.data_ptr(), v.data_ptr(), n, e,
                                                    pipe.idx.data_ptr(), pipe.val.data_ptr(), bpc,
                                                    sink.data_ptr(), s), "ceil_read3_write")
            mix = ms if mix is None or ms < mix else mix
            del sink
        b = 12 * n + 10 * e
        out["read_then_write"] = {"ms": rd + wr, "read_ms": rd, "write_ms": wr,
                                  "gbs": b / ((rd + wr) / 1e3) / 1e9, "bytes": b, "entries": e,
                                  "naive_mix_ms": mix}
    R = len(pipe.shards)
    if R <= 16:
        scratch = [torch.empty_like(t) for t in pipe.shards]
        arr = lambda T, xs: (T * R)(*xs)                # noqa: E731
        dst = arr(ctypes.c_void_p, [t.data_ptr() for t in scratch])
        off = arr(ctypes.c_void_p, [t.data_ptr() for t in pipe.off])
        cap = arr(ctypes.c_int64, pipe.rank_capacity)
        numel = arr(ctypes.c_int64, [t.numel() for t in pipe.shards])
        best = None
        for bpc in (4, 8, 16):
            ms = timed(lambda: lib.ceil_line_writes(R, dst, off, pipe.rank_count.data_ptr(), cap,
                                                    numel, bpc, s), "ceil_line_writes")
            best = ms if best is None or ms < best else best
        out["apply_scattered_lines"] = {"ms": best}
        del scratch
    torch.cuda.empty_cache()
    return out


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


def _stats(xs):
    xs = sorted(xs)
    k = len(xs)
    med = xs[k // 2] if k % 2 else 0.5 * (xs[k // 2 - 1] + xs[k // 2])
    return {"mean": sum(xs) / k, "median": med, "min": xs[0], "max": xs[-1]}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="qwen3_8b_tp4")
    ap.add_argument("--lr", type=float, default=None)
    ap.add_argument("--literal", action="store_true",
                    help="literal operation order of the AdamW inverse (four divisions)")
    ap.add_argument("--ordered", action="store_true",
                    help="dte_extract_delta_ordered (ascending, deterministic delta)")
    ap.add_argument("--norm-group", action="store_true",
                    help="norms in a parameter group without weight decay")
    ap.add_argument("--capacity-fraction", type=float, default=None,
                    help="delta buffer size as a fraction of the elements (default 0.02, "
                         "0.25 for the learning-rate sweep)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-procs", type=int, default=0,
                    help="processes of the oracle's pool run (default: the usable cores)")
    ap.add_argument("--no-ceilings", action="store_true",
                    help="skip the reference read-stream and scattered-line measurements")
    ap.add_argument("--flush-gb", type=float, default=None, metavar="GB",
                    help="touch this many GB (read and write) before every timed step, "
                         "outside the step's own events (default: 1 GB when theta, m, v "
                         "occupy less than 2 GB, so that they cannot stay in the 256 MB "
                         "last-level cache between steps; else 0)")
    ap.add_argument("--settle", type=float, default=15.0, metavar="SECONDS",
                    help="wait before allocating the state (after the CPU baseline, which "
                         "runs first): device memory that a process "
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

    cpu, cpu_s = None, 0.0
    if not args.no_cpu_baseline and args.copy_calibration <= 0:
        # before any GPU work: the oracle's worker processes are forked from a
        # process that has not initialised the GPU
        log("bench: timing the CPU oracle")
        t = time.perf_counter()
        cpu = cpu_baseline(args.cpu_procs)
        cpu_s = time.perf_counter() - t
        log("bench: CPU oracle done in %.1f s" % cpu_s)

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
    settle = args.settle
    if settle > 0:
        log("bench: settling %.0f s before allocating" % settle)
        time.sleep(settle)
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
    flush_gb = args.flush_gb if args.flush_gb is not None else (1.0 if 12 * n < 2e9 else 0.0)
    flush = (torch.zeros(int(flush_gb * 1e9) // 8, dtype=torch.float32, device="cuda")
             if flush_gb > 0 else None)

    # events per step: 0 step start (before the cursor reset), 1 extract
    # start, 2 extract end, 3 remap end, 4 apply end
    def step(ev=None):
        rec = (lambda i: ev[i].record(stream)) if ev else (lambda i: None)
        rec(0)
        if apply_only:
            rec(1)
            rec(2)
            rec(3)
            pipe.apply()
            rec(4)
            return
        pipe.reset()
        rec(1)
        if len(runs) == 1:
            pipe.extract(p, m, v, hp)
        else:
            pipe.extract_runs(p, m, v, runs)
        rec(2)
        pipe.remap()
        rec(3)
        pipe.apply()
        rec(4)

    if apply_only:                           # delta and buckets prepared untimed
        pipe.step(p, m, v, hp)
    for _ in range(args.warmup):
        if flush is not None:
            flush.add_(1.0)
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for k in range(args.steps):
        if flush is not None:
            flush.add_(1.0)                  # reads and writes flush_gb GB, outside the step
        step(evs[k])
    end.record(stream)
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    per_step = [e[0].elapsed_time(e[4]) for e in evs]
    # with a cache flush between steps the step time is the steps' own
    # events; else the whole bracketed interval
    ms_step = sum(per_step) / args.steps if flush is not None else total_ms / args.steps
    changed = int(pipe.cursor.item())
    counts = pipe.rank_count.cpu().tolist()
    routed = int(sum(counts))
    if changed > cap or any(c > cap for c in counts):
        log("bench: capacity exceeded (changed %d, capacity %d)" % (changed, cap))
        return 3
    c = changed / n
    ext = _stats([e[1].elapsed_time(e[2]) for e in evs])
    rem = _stats([e[2].elapsed_time(e[3]) for e in evs])
    app = _stats([e[3].elapsed_time(e[4]) for e in evs])

    if apply_only:
        k = app
        k_bytes = routed * (8 + 2 + 2)       # read offset + value, write value
        value = routed / (ms_step / 1e3)
        metric_unit = "entries/s"
        kernel = "apply"
    else:
        k = ext
        k_bytes = 12 * n + 10 * changed       # read theta, m, v; write (idx, val)
        value = n / (ms_step / 1e3)
        metric_unit = "elements/s"
        kernel = "extract"
    if apply_only:
        step_bytes = k_bytes
    else:
        step_bytes = 12 * n + 10 * changed + 10 * changed + 10 * routed + 12 * routed
    achieved = k_bytes / (k["mean"] / 1e3) / 1e9
    # the counters were taken for the default configuration only (folded
    # order, unordered output, one parameter group)
    default_mode = not (args.ordered or args.literal or args.norm_group)
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
        "config": {"workload": wl.name, "elements": n, "changed": changed,
                   "extract_calls": len(runs), "settle_s": settle, "ordered": ordered,
                   "order": "literal" if args.literal else "folded",
                   "change_fraction": c, "receiver_ranks": len(counts),
                   "routed_entries": routed, "lr": hp.lr,
                   "step_algorithmic_bytes": step_bytes,
                   "step_gbs": step_bytes / (ms_step / 1e3) / 1e9,
                   "step_frac_of_hbm_peak": step_bytes / (ms_step / 1e3) / 1e9 / HBM_PEAK_GBS,
                   "flush_gb_between_steps": flush_gb},
        "timing": {"step_ms": _stats(per_step), "bracket_ms_per_step": total_ms / args.steps,
                   "extract_ms": ext, "remap_ms": rem, "apply_ms": app},
        "roofline": {"kernel": kernel, "bound": "hbm", "achieved": achieved,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": (measured_traffic(wl.name, kernel, "unordered")
                                 if default_mode else None),
                     "kernel_ms": k["mean"], "kernel_ms_median": k["median"],
                     "bytes_per_launch": k_bytes},
    }
    if not apply_only:
        out["config"].update({"extract_ms": ext["mean"], "remap_ms": rem["mean"],
                              "apply_ms": app["mean"]})
    if not args.no_ceilings:
        log("bench: reference read stream and scattered lines")
        ce = ceilings(p, m, v, pipe, stream, 0 if apply_only else changed,
                      touch=(lambda: flush.add_(1.0)) if flush is not None else None)
        rs = ce["read_stream"]
        if kernel == "extract":
            rs["kernel_frac"] = achieved / rs["gbs"]
            if "read_then_write" in ce:
                ce["read_then_write"]["kernel_frac"] = ce["read_then_write"]["ms"] / k["mean"]
        if "apply_scattered_lines" in ce:
            ce["apply_scattered_lines"]["apply_ms"] = app["mean"]
            ce["apply_scattered_lines"]["apply_frac"] = \
                ce["apply_scattered_lines"]["ms"] / app["mean"]
        out["roofline"]["ceilings"] = ce
    if flush is not None:
        del flush
        torch.cuda.empty_cache()
    if args.store and not apply_only:
        out["storage"] = storage_leg(args.store, wl, spec, p, m, v, hp, cap)
    del p, m, v
    pipe.close()
    torch.cuda.empty_cache()
    if cpu is not None:
        out["cpu_baseline"] = cpu
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
