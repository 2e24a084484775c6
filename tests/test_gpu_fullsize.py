"""Full-size GPU parity on the real workload shapes, in the launch
configuration bench.py times (same entry points, same delta capacity).

The oracle computes the complete delta of each workload on the host cores
(about 30 s for the 8.19e9-element Qwen3-8B state on 16 cores), so the
delta index set, BF16 values and every receiver bucket are compared
exactly.  Applied shards (tens of GB) are checked by gathering the GPU
shard at every offset of the oracle's buckets, plus the property that the
number of written elements equals the routed count (shards start at a
pattern the delta never contains).  Reconstructed weights are compared at
0 ulp on windows of every kind of tensor.
"""
import sys

import numpy as np
import pytest
import torch

import synth
from oracle import plan as oplan
from oracle import remap as oremap
from oracle import run as orun
from paper_2608_00455_amd import layouts
from paper_2608_00455_amd.pipeline import DeltaPipeline, generate_state
from synth import workloads as W

pytestmark = pytest.mark.gpu

SENTINEL = 0x7FFF      # a NaN pattern that BF16 rounding never produces


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def sync():
    torch.cuda.synchronize()


def sentinel_shards(spec):
    return [torch.full((n,), SENTINEL, dtype=torch.int16, device="cuda") for n in spec.rank_numel]


def golden_diag(name):
    import json
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "diagnostics.json")
    return json.load(open(path))["workloads"][name]


def check_oracle_diag(wl, res):
    g = golden_diag(wl.name)
    d = res.diag
    assert (d.n, d.changed, d.bf16_recon_mismatch, d.fp32_recon_mismatch) == \
        (g["elements"], g["changed"], g["bf16_recon_mismatch"], g["fp32_recon_mismatch"])


def check_delta(pipe, res):
    idx, val, total = pipe.delta()
    assert total == res.idx.size, (total, res.idx.size)
    assert np.array_equal(idx, res.idx)
    assert np.array_equal(val, res.val)


def check_buckets_and_shards(pipe, pl, want):
    buckets, counts = pipe.buckets()
    for r in range(pl.nranks):
        assert counts[r] == want[r][0].size, (r, counts[r], want[r][0].size)
        assert np.array_equal(buckets[r][0], want[r][0]), r
        assert np.array_equal(buckets[r][1], want[r][1]), r
        shard = pipe.shards[r]
        written = int((shard != SENTINEL).sum().item())
        assert written == want[r][0].size, (r, written)
        if want[r][0].size:
            got = shard[torch.from_numpy(want[r][0]).cuda()].cpu().numpy().view(np.uint16)
            assert np.array_equal(got, want[r][1]), r


def check_theta_hat_windows(wl, p, m, v, spec, picks):
    """0-ulp reconstructed weights on windows (tensor index, start, length)."""
    begins = wl.flat_begins()
    wins = [orun.Window(k, lo, min(wl.tensors[k].numel, lo + n)) for k, lo, n in picks]
    res = orun.extract(wl, wins=wins, keep=("ph",))
    pipe = DeltaPipeline(spec, capacity=1 << 22)
    for part in res.parts:
        w = part.window
        a = begins[w.tensor] + w.lo
        n = w.hi - w.lo
        prev = torch.empty(n, dtype=torch.float32, device="cuda")
        pipe.reset()
        pipe.extract(p[a:a + n], m[a:a + n], v[a:a + n], wl.hp, index_base=a, out_prev=prev)
        sync()
        assert np.array_equal(prev.cpu().numpy().view(np.uint32), part.ph.view(np.uint32)), w
        idx, val, _ = pipe.delta()
        assert np.array_equal(idx, part.idx) and np.array_equal(val, part.val), w
    pipe.close()


def pick_windows(wl, seed, count=6, length=1 << 20):
    """The first and last elements of the shard, every small tensor of the
    first layer, and seeded windows in large tensors."""
    rng = np.random.default_rng(seed)
    last = len(wl.tensors) - 1
    picks = [(0, 0, length), (last, max(0, wl.tensors[last].numel - length), length)]
    first_layer = [k for k, t in enumerate(wl.tensors) if t.layer == 0 and t.numel <= 1 << 16]
    picks += [(k, 0, wl.tensors[k].numel) for k in first_layer]
    big = [k for k, t in enumerate(wl.tensors) if t.numel > length]
    for k in rng.choice(big, size=count, replace=False):
        lo = int(rng.integers(0, wl.tensors[k].numel - length))
        picks.append((int(k), lo, length))
    return picks


@pytest.fixture(scope="module")
def qwen3_8b():
    wl = W.qwen3_8b(4)
    say("fullsize: oracle over %s (%d elements)" % (wl.name, wl.numel))
    res = orun.extract(wl)
    say("fullsize: oracle done, %d changed, %s" % (res.idx.size, res.diag))
    check_oracle_diag(wl, res)
    p, m, v = generate_state(wl)
    yield wl, res, p, m, v
    del p, m, v
    torch.cuda.empty_cache()


def test_qwen3_8b_tp4_full(qwen3_8b):
    wl, res, p, m, v = qwen3_8b
    spec = layouts.build_spec(wl)
    pl = oplan.build_plan(wl)
    pipe = DeltaPipeline(spec, capacity=int(wl.numel * 0.02), shards=sentinel_shards(spec))
    pipe.step(p, m, v, wl.hp)
    sync()
    check_delta(pipe, res)
    say("fullsize: delta equal; remapping with the oracle")
    check_buckets_and_shards(pipe, pl, oremap.remap(pl, res.idx, res.val))
    pipe.close()
    del pipe
    torch.cuda.empty_cache()
    check_theta_hat_windows(wl, p, m, v, spec, pick_windows(wl, 1))


def test_qwen3_8b_ordered_full(qwen3_8b):
    """Ordered extract at full size: the raw output is the oracle's sorted
    delta, entry for entry."""
    wl, res, p, m, v = qwen3_8b
    spec = layouts.build_spec(wl)
    pipe = DeltaPipeline(spec, capacity=int(wl.numel * 0.02), ordered=True)
    pipe.reset()
    pipe.extract(p, m, v, wl.hp)
    sync()
    idx, val, total = pipe.delta(raw=True)
    assert total == res.idx.size
    assert np.array_equal(idx, res.idx)
    assert np.array_equal(val, res.val)
    pipe.close()
    del pipe
    torch.cuda.empty_cache()


def test_qwen3_8b_store_round_trip_full(qwen3_8b, tmp_path):
    """The full Qwen3-8B delta published from the device (ordered extract,
    zstd chunks) and read back into device memory equals the oracle's."""
    import time
    from paper_2608_00455_amd import store as S
    wl, res, p, m, v = qwen3_8b
    spec = layouts.build_spec(wl)
    pipe = DeltaPipeline(spec, capacity=int(wl.numel * 0.02), ordered=True)
    pipe.reset()
    pipe.extract(p, m, v, wl.hp)
    segs = S.segments_of([t.name for t in wl.tensors], wl.flat_begins(),
                         [t.numel for t in wl.tensors])
    opt = S.Options(threads=16)
    t0 = time.perf_counter()
    st = S.write_part_device(tmp_path, 1, 0, segs, pipe.idx.data_ptr(), pipe.val.data_ptr(),
                             pipe.cursor.data_ptr(), pipe.capacity, opt)
    assert S.commit(tmp_path, 1, 0, 1)
    t1 = time.perf_counter()
    pipe.idx.fill_(-1)
    n, _ = S.read_device(tmp_path, 1, 0, pipe.idx.data_ptr(), pipe.val.data_ptr(), pipe.capacity,
                         threads=16)
    t2 = time.perf_counter()
    say("fullsize: store %d entries, %d chunks, %.1f MB raw, %.1f MB stored, publish %.2f s, "
        "read %.2f s" % (st.entries, st.chunks, st.raw_bytes / 1e6, st.stored_bytes / 1e6,
                         t1 - t0, t2 - t1))
    assert n == res.idx.size == st.entries
    pipe.cursor.fill_(n)
    idx, val, _ = pipe.delta(raw=True)
    assert np.array_equal(idx, res.idx) and np.array_equal(val, res.val)
    pipe.close()
    del pipe
    torch.cuda.empty_cache()


def test_qwen3_8b_fused_extract_remap_full(qwen3_8b):
    """dte_extract_remap at full size: buckets and applied shards equal the
    oracle's remap of its complete delta."""
    wl, res, p, m, v = qwen3_8b
    spec = layouts.build_spec(wl)
    pl = oplan.build_plan(wl)
    pipe = DeltaPipeline(spec, capacity=1, rank_capacity=[int(wl.numel * 0.006)] * 4,
                         shards=sentinel_shards(spec))
    pipe.step_fused(p, m, v, wl.hp)
    sync()
    assert int(pipe.cursor.item()) == res.idx.size
    check_buckets_and_shards(pipe, pl, oremap.remap(pl, res.idx, res.val))
    pipe.close()
    del pipe
    torch.cuda.empty_cache()


def test_qwen3_8b_tp8_apply_full(qwen3_8b):
    """The Qwen3-8B delta remapped to eight TP=8 receivers and applied."""
    wl, res, p, m, v = qwen3_8b
    wl8 = W.qwen3_8b(8)
    spec8 = layouts.build_spec(wl8)
    pl8 = oplan.build_plan(wl8)
    pipe = DeltaPipeline(spec8, capacity=int(wl.numel * 0.02), shards=sentinel_shards(spec8))
    pipe.step(p, m, v, wl.hp)
    sync()
    check_delta(pipe, res)
    check_buckets_and_shards(pipe, pl8, oremap.remap(pl8, res.idx, res.val))
    pipe.close()


def test_qwen3_30b_a3b_share_full():
    wl = W.qwen3_30b_a3b_share(synth.word)
    say("fullsize: oracle over %s (%d elements)" % (wl.name, wl.numel))
    res = orun.extract(wl)
    say("fullsize: oracle done, %d changed, %s" % (res.idx.size, res.diag))
    check_oracle_diag(wl, res)
    # untouched experts (zero moments) never change
    begins = wl.flat_begins()
    for k, t in enumerate(wl.tensors):
        if not t.touched:
            lo = np.searchsorted(res.idx, begins[k])
            hi = np.searchsorted(res.idx, begins[k] + t.numel)
            assert lo == hi, t.name
    p, m, v = generate_state(wl)
    spec = layouts.build_spec(wl)
    pl = oplan.build_plan(wl)
    pipe = DeltaPipeline(spec, capacity=int(wl.numel * 0.02), shards=sentinel_shards(spec))
    pipe.step(p, m, v, wl.hp)
    sync()
    check_delta(pipe, res)
    check_buckets_and_shards(pipe, pl, oremap.remap(pl, res.idx, res.val))
    pipe.close()
    del pipe
    torch.cuda.empty_cache()
    check_theta_hat_windows(wl, p, m, v, spec, pick_windows(wl, 3))
    del p, m, v
    torch.cuda.empty_cache()


@pytest.mark.parametrize("lr", W.SWEEP_LR)
def test_qwen3_8b_layers_lr_sweep_full(lr):
    wl = W.qwen3_8b_layers_sweep(lr)
    say("fullsize: sweep lr %g" % lr)
    res = orun.extract(wl)
    check_oracle_diag(wl, res)
    p, m, v = generate_state(wl)
    spec = layouts.build_spec(wl)
    pl = oplan.build_plan(wl)
    pipe = DeltaPipeline(spec, capacity=int(wl.numel * 0.25), shards=sentinel_shards(spec))
    pipe.step(p, m, v, wl.hp)
    sync()
    check_delta(pipe, res)
    check_buckets_and_shards(pipe, pl, oremap.remap(pl, res.idx, res.val))
    pipe.close()
    del pipe, p, m, v
    torch.cuda.empty_cache()


@pytest.mark.parametrize("rank", [1])
def test_qwen3_8b_layers_mcore_full(rank):
    """Four Qwen3-8B layers held as trainer TP rank `rank` of 2 in the
    Megatron-Core layout, sent to four TP=4 receivers.  The oracle detects
    in the paper's order (MCore inversion, conversion, canonical BF16
    comparison) and routes through the canonical plan."""
    from oracle import mcore
    wl = W.qwen3_8b_layers_mcore(trainer_rank=rank)
    say("fullsize: mcore oracle over %s" % wl.name)
    want = mcore.extract(wl)
    ci = mcore.canonical_index(wl)
    say("fullsize: mcore oracle done, %d changed of %d" % (want.idx.size, ci.size))
    twin = W.canonical_twin(wl)
    cplan = oplan.build_plan(twin)
    p, m, v = generate_state(wl)
    spec = layouts.build_spec(wl)
    assert spec.total == ci.size == p.numel()
    pipe = DeltaPipeline(spec, capacity=int(ci.size * 0.02), shards=sentinel_shards(spec))
    pipe.step(p, m, v, wl.hp)
    sync()
    idx, val, total = pipe.delta()
    assert total == want.idx.size
    mapped = ci[idx]
    order = np.argsort(mapped, kind="stable")
    assert np.array_equal(mapped[order], want.idx)
    assert np.array_equal(val[order], want.val)
    check_buckets_and_shards(pipe, cplan, oremap.remap(cplan, want.idx, want.val))
    pipe.close()
    del pipe, p, m, v
    torch.cuda.empty_cache()


def test_qwen3_8b_layers_literal_order_full():
    """Four Qwen3-8B layers at lr 1e-4 (DECAY != 1, 14 % changed) with the
    literal operation order of eq. adamw_inverse, forward step included."""
    wl = W.qwen3_8b_layers_sweep(1e-4)
    hp = W.StepHP(lr=1e-4, order=W.ORDER_LITERAL)
    say("fullsize: literal order")
    res = orun.extract(wl, hp=hp)
    p, m, v = generate_state(wl, hp)
    spec = layouts.build_spec(wl)
    pl = oplan.build_plan(wl)
    pipe = DeltaPipeline(spec, capacity=int(wl.numel * 0.25), shards=sentinel_shards(spec))
    pipe.step(p, m, v, hp)
    sync()
    check_delta(pipe, res)
    check_buckets_and_shards(pipe, pl, oremap.remap(pl, res.idx, res.val))
    pipe.close()
    del pipe, p, m, v
    torch.cuda.empty_cache()
