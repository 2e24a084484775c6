"""Pins of the oracle's transfer plan and remap (sec. 4.2.2).

The remap of every canonical flat offset must reproduce the dense receiver
route (tests/dense_route.py) exactly: this shows the plan's unravel /
containment / ravel is a bijection from (canonical element, replica) onto
the receiver elements.  Sizes of the real workloads are checked against
their shape arithmetic.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import plan as oplan
from oracle import remap as oremap
from synth import workloads as W

from dense_route import dense_receivers

SMALL = [
    lambda: W.tiny_block(),
    lambda: W.scaled_dense(layers=2, tp=2),
    lambda: W.scaled_dense(layers=1, tp=4, heads_kv=4, heads_q=8),
    lambda: W.scaled_dense(layers=1, tp=8, heads_kv=8, heads_q=8, head_dim=16, hidden=64,
                           intermediate=128, vocab=64),
    lambda: W.scaled_moe(synth.word, layers=2, ranks=4, attn_tp=2, experts=8),
    lambda: W.scaled_moe(synth.word, layers=1, ranks=8, attn_tp=2, experts=16, hidden=64,
                         head_dim=16, expert_intermediate=24),
]


@pytest.mark.parametrize("make", SMALL)
def test_remap_of_all_offsets_equals_dense_route(make):
    wl = make()
    pl = oplan.build_plan(wl)
    n = wl.numel
    tags = np.arange(n, dtype=np.int64)
    buckets = oremap.remap(pl, tags, tags)
    want = dense_receivers(wl, torch.from_numpy(tags))
    assert len(buckets) == len(want) == pl.nranks
    for r, (off, tag) in enumerate(buckets):
        assert want[r].numel() == pl.rank_numel[r]
        # every receiver element written exactly once
        assert np.array_equal(off, np.arange(pl.rank_numel[r]))
        assert np.array_equal(tag, want[r].numpy())


def _replication(wl, pl):
    vol = np.zeros(len(wl.tensors), np.int64)
    for o in pl.ops:
        vol[o.segment] += int(np.prod(o.extent))
    return vol


@pytest.mark.parametrize("make,ranks,rank_numel,nseg,nops", [
    (lambda: W.tiny_block(), 2, 5_638_144, 9, 18),
    (lambda: W.qwen3_8b(4), 4, 2_047_915_008, 399, 1596),
    (lambda: W.qwen3_8b(8), 8, 1_024_111_616, 399, 3192),
    (lambda: W.qwen3_30b_a3b_share(synth.word), 8, 1_022_413_824, 4716, 5472),
    # per layer: 8,448 replicated norm elements, the rest split four ways
    (lambda: W.qwen3_8b_layers_sweep(1e-6), 4, 4 * ((192_946_432 - 8448) // 4 + 8448), 44, 176),
])
def test_real_workload_plan_sizes(make, ranks, rank_numel, nseg, nops):
    wl = make()
    pl = oplan.build_plan(wl)
    assert pl.nranks == ranks
    assert len(pl.seg_begin) == nseg and len(pl.ops) == nops
    assert all(x == rank_numel for x in pl.rank_numel)
    # receiver elements = sum over segments of numel * replication
    vol = _replication(wl, pl)
    assert vol.sum() == sum(pl.rank_numel)
    numel = np.array([t.numel for t in wl.tensors], np.int64)
    assert np.all(vol % numel == 0) and np.all(vol >= numel)


def test_oracle_remap_on_one_to_four_dimensional_segments_by_brute_force():
    """The oracle's remap (numpy unravel / ravel) against coordinates worked
    out by repeated division and Horner's rule, one element at a time, on a
    sample of every segment of a plan with 1-D to 4-D segments."""
    from highdim_plan import HighDimSpec
    from oracle import remap as oremap
    spec = HighDimSpec()
    pl = spec.oracle_plan
    rng = np.random.default_rng(26080455 + 43)
    idx = np.unique(np.concatenate([
        rng.integers(b, b + int(np.prod(s)), 400) for b, s in zip(pl.seg_begin, pl.seg_shape)]))
    val = (idx % 65521).astype(np.uint16)
    got = oremap.remap(pl, idx, val)
    want = [dict() for _ in range(pl.nranks)]
    for i, x in zip(idx.tolist(), val.tolist()):
        s = max(k for k, b in enumerate(pl.seg_begin) if b <= i)
        rest = i - pl.seg_begin[s]
        shape = pl.seg_shape[s]
        u = [0] * len(shape)
        for d in range(len(shape) - 1, -1, -1):
            rest, u[d] = divmod(rest, shape[d])
        for o in pl.ops:
            if o.segment != s:
                continue
            if all(o.src_origin[d] <= u[d] < o.src_origin[d] + o.extent[d]
                   for d in range(len(shape))):
                j = 0
                for d in range(len(shape)):
                    j = j * o.dst_shape[d] + (u[d] - o.src_origin[d] + o.dst_origin[d])
                assert o.dst_base + j not in want[o.rank]
                want[o.rank][o.dst_base + j] = x
    for r in range(pl.nranks):
        keys = sorted(want[r])
        assert np.array_equal(got[r][0], np.array(keys, dtype=np.int64))
        assert np.array_equal(got[r][1], np.array([want[r][k] for k in keys], dtype=np.uint16))
