"""Degenerate calls the C ABI allows: zero capacities with NULL output
pointers (count-only calls).  The counts must equal the oracle's (sec.
4.2.1 detection, sec. 4.2.2 remap) and nothing may be written."""
import sys

import numpy as np
import pytest
import torch

from oracle import plan as oplan
from oracle import remap as oremap
from oracle import run as orun
from paper_2608_00455_amd import binding as B
from paper_2608_00455_amd import layouts
from paper_2608_00455_amd.pipeline import Plan
from synth import workloads as W

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def case():
    wl = W.scaled_dense(layers=1, tp=2, lr=1e-4)
    res = orun.extract(wl, keep=("p", "m", "v"))
    st = {k: orun.flat(res.parts, k) for k in ("p", "m", "v")}
    dev = {k: torch.from_numpy(np.ascontiguousarray(x)).cuda() for k, x in st.items()}
    return wl, res, dev


def test_count_only_extract_unordered_and_ordered(case):
    wl, res, d = case
    say("case: count-only extract", res.idx.size)
    assert res.idx.size > 0
    s = torch.cuda.current_stream().cuda_stream
    cur = torch.zeros(1, dtype=torch.int64, device="cuda")
    B.dte_extract_delta(d["p"].data_ptr(), d["m"].data_ptr(), d["v"].data_ptr(), wl.numel, 0,
                        wl.hp, 0, 0, 0, cur.data_ptr(), 0, s)
    torch.cuda.synchronize()
    assert int(cur.item()) == res.idx.size
    ws = torch.empty(max(1, B.dte_ordered_workspace_bytes(0)), dtype=torch.uint8, device="cuda")
    cur.zero_()
    B.dte_extract_delta_ordered(d["p"].data_ptr(), d["m"].data_ptr(), d["v"].data_ptr(),
                                wl.numel, 0, wl.hp, 0, 0, 0, cur.data_ptr(), ws.data_ptr(),
                                ws.numel(), 0, s)
    torch.cuda.synchronize()
    assert int(cur.item()) == res.idx.size


def test_rank_without_bucket_is_counted_not_written(case):
    wl, res, d = case
    say("case: remap with a zero-capacity rank")
    spec = layouts.build_spec(wl)
    plan = Plan(spec)
    want = oremap.remap(oplan.build_plan(wl), res.idx, res.val)
    s = torch.cuda.current_stream().cuda_stream
    m = res.idx.size
    idx = torch.from_numpy(res.idx).cuda()
    val = torch.from_numpy(res.val.view(np.int16)).cuda()
    count = torch.tensor([m], dtype=torch.int64, device="cuda")
    cap = [m, 0]
    off0 = torch.full((m,), -7, dtype=torch.int64, device="cuda")
    val0 = torch.zeros(m, dtype=torch.int16, device="cuda")
    rank_count = torch.zeros(2, dtype=torch.int64, device="cuda")
    shards = [torch.full((n,), 0x55, dtype=torch.int16, device="cuda") for n in spec.rank_numel]
    B.dte_remap(plan.handle, idx.data_ptr(), val.data_ptr(), count.data_ptr(), m,
                [off0.data_ptr(), 0], [val0.data_ptr(), 0], cap, rank_count.data_ptr(), s)
    B.dte_apply(plan.handle, [t.data_ptr() for t in shards], [off0.data_ptr(), 0],
                [val0.data_ptr(), 0], rank_count.data_ptr(), cap, s)
    torch.cuda.synchronize()
    counts = rank_count.cpu().tolist()
    assert counts == [want[0][0].size, want[1][0].size]
    got = off0[:counts[0]].cpu().numpy()
    order = got.argsort(kind="stable")
    assert np.array_equal(got[order], want[0][0])
    assert np.array_equal(val0[:counts[0]].cpu().numpy().view(np.uint16)[order], want[0][1])
    assert bool((shards[1] == 0x55).all())           # rank 1 has no bucket: untouched
    plan.close()


def test_fused_call_with_no_buckets_counts_every_rank(case):
    wl, res, d = case
    say("case: fused count-only")
    spec = layouts.build_spec(wl)
    plan = Plan(spec)
    want = oremap.remap(oplan.build_plan(wl), res.idx, res.val)
    s = torch.cuda.current_stream().cuda_stream
    cur = torch.zeros(1, dtype=torch.int64, device="cuda")
    rank_count = torch.zeros(spec.nranks, dtype=torch.int64, device="cuda")
    B.dte_extract_remap(d["p"].data_ptr(), d["m"].data_ptr(), d["v"].data_ptr(), wl.numel, 0,
                        wl.hp, plan.handle, [0] * spec.nranks, [0] * spec.nranks,
                        [0] * spec.nranks, rank_count.data_ptr(), cur.data_ptr(), s)
    torch.cuda.synchronize()
    assert int(cur.item()) == res.idx.size
    assert rank_count.cpu().tolist() == [w[0].size for w in want]
    plan.close()


def test_entries_outside_the_plan_or_shard_are_ignored(case):
    """remap skips offsets outside [0, total) (include/dte.h); apply skips
    bucket offsets outside a shard."""
    wl, res, d = case
    say("case: out-of-range entries")
    spec = layouts.build_spec(wl)
    plan = Plan(spec)
    total = spec.total
    rng = np.random.default_rng(26080455 + 91)
    bad = np.array([-1, -(1 << 40), total, total + 1, 1 << 50, -total], np.int64)
    idx = np.concatenate([res.idx, bad])
    val = np.concatenate([res.val, np.full(bad.size, 0xBEEF, np.uint16)])
    perm = rng.permutation(idx.size)
    idx, val = idx[perm], val[perm]
    want = oremap.remap(oplan.build_plan(wl), res.idx, res.val)
    s = torch.cuda.current_stream().cuda_stream
    m = idx.size
    d_idx = torch.from_numpy(idx).cuda()
    d_val = torch.from_numpy(val.view(np.int16)).cuda()
    count = torch.tensor([m], dtype=torch.int64, device="cuda")
    off = [torch.empty(m, dtype=torch.int64, device="cuda") for _ in range(spec.nranks)]
    rv = [torch.empty(m, dtype=torch.int16, device="cuda") for _ in range(spec.nranks)]
    rank_count = torch.zeros(spec.nranks, dtype=torch.int64, device="cuda")
    B.dte_remap(plan.handle, d_idx.data_ptr(), d_val.data_ptr(), count.data_ptr(), m,
                [t.data_ptr() for t in off], [t.data_ptr() for t in rv], [m] * spec.nranks,
                rank_count.data_ptr(), s)
    torch.cuda.synchronize()
    counts = rank_count.cpu().tolist()
    for r in range(spec.nranks):
        assert counts[r] == want[r][0].size, r
        got = off[r][:counts[r]].cpu().numpy()
        order = got.argsort(kind="stable")
        assert np.array_equal(got[order], want[r][0]), r
        assert np.array_equal(rv[r][:counts[r]].cpu().numpy().view(np.uint16)[order],
                              want[r][1]), r
    # apply: buckets with offsets outside the shard
    numel = spec.rank_numel
    b_off = [np.array([0, -1, numel[r] - 1, numel[r], -(1 << 40), 1 << 45, 5], np.int64)
             for r in range(spec.nranks)]
    b_val = [np.arange(7, dtype=np.uint16) + 100 * (r + 1) for r in range(spec.nranks)]
    shards = [torch.full((n,), 0x33, dtype=torch.int16, device="cuda") for n in numel]
    dt_off = [torch.from_numpy(x).cuda() for x in b_off]
    dt_val = [torch.from_numpy(x.view(np.int16)).cuda() for x in b_val]
    cnt = torch.tensor([7] * spec.nranks, dtype=torch.int64, device="cuda")
    B.dte_apply(plan.handle, [t.data_ptr() for t in shards], [t.data_ptr() for t in dt_off],
                [t.data_ptr() for t in dt_val], cnt.data_ptr(), [7] * spec.nranks, s)
    torch.cuda.synchronize()
    for r in range(spec.nranks):
        expect = np.full(numel[r], 0x33, np.uint16)
        for o, v in zip(b_off[r], b_val[r]):
            if 0 <= o < numel[r]:
                expect[o] = v
        assert np.array_equal(shards[r].cpu().numpy().view(np.uint16), expect), r
    plan.close()
