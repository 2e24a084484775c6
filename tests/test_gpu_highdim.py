"""GPU parity of remap, apply and the fused call on plans whose segments
have one to four dimensions (the plan format allows four; the model
workloads only use vectors and matrices).

The plan is written out here twice, as the oracle's Plan and as the C-ABI
structs; the oracle's remap (sec. 4.2.2) is the reference.  Inputs are
seeded synthetic draws; the post-step state comes from the oracle's
forward step.
"""
import sys

import numpy as np
import pytest
import torch

from highdim_plan import HighDimSpec
from oracle import core as ocore
from oracle import remap as oremap
from paper_2608_00455_amd.pipeline import DeltaPipeline
from synth import workloads as W

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host_u16(t):
    return t.cpu().numpy().view(np.uint16)


def check_buckets(pipe, spec, want, old):
    torch.cuda.synchronize()
    buckets, counts = pipe.buckets()
    expect = oremap.apply([x.copy() for x in old], want)
    for r in range(spec.nranks):
        assert counts[r] == want[r][0].size, r
        assert np.array_equal(buckets[r][0], want[r][0]), r
        assert np.array_equal(buckets[r][1], want[r][1]), r
        assert np.array_equal(host_u16(pipe.shards[r]), expect[r]), r


def _pipe(spec, capacity, old):
    return DeltaPipeline(spec, capacity=capacity,
                         rank_capacity=[max(1, n) for n in spec.rank_numel],
                         shards=[dev(x.view(np.int16)) for x in old])


@pytest.mark.parametrize("pattern", ["all", "ascending", "shuffled"])
def test_remap_apply_segments_of_one_to_four_dimensions(pattern):
    """Remap of every offset, of an ascending subset and of a shuffled
    subset (chunks that span segments, in any order) equals the oracle's."""
    spec = HighDimSpec()
    n = spec.numel
    rng = np.random.default_rng(26080455 + 41)
    if pattern == "all":
        idx = np.arange(n, dtype=np.int64)
    else:
        idx = np.flatnonzero(rng.random(n) < 0.3).astype(np.int64)
        if pattern == "shuffled":
            rng.shuffle(idx)
    val = rng.integers(0, 1 << 16, idx.size, dtype=np.uint16)
    say("case: high-dimensional remap", pattern, idx.size)
    old = [np.full(k, 0x7FFF, np.uint16) for k in spec.rank_numel]
    want = oremap.remap(spec.oracle_plan, idx, val)
    pipe = _pipe(spec, idx.size, old)
    pipe.idx[:idx.size].copy_(dev(idx))
    pipe.val[:idx.size].copy_(dev(val.view(np.int16)))
    pipe.cursor.fill_(idx.size)
    pipe.remap()
    pipe.apply()
    check_buckets(pipe, spec, want, old)
    pipe.close()


@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("lr", [1e-5, 1e-3])
def test_extract_paths_on_high_dimensional_plan(lr, fused):
    """extract + remap + apply, and the fused call, over the whole plan on a
    seeded post-step state, against oracle detection and remap."""
    spec = HighDimSpec()
    n = spec.numel
    hp = W.StepHP(lr=lr)
    sc = ocore.derive_scalars(hp)
    rng = np.random.default_rng(26080455 + 42)
    p_prev = (0.02 * rng.standard_normal(n)).astype(np.float32)
    m_prev = (1e-4 * rng.standard_normal(n)).astype(np.float32)
    v_prev = np.abs(1e-6 * rng.standard_normal(n)).astype(np.float32)
    g = (1e-3 * rng.standard_normal(n)).astype(np.float32)
    p, m, v = ocore.adamw_forward(p_prev, m_prev, v_prev, g, sc)
    idx, val, ph = ocore.detect(p, m, v, sc)
    say("case: high-dimensional extract", lr, "fused" if fused else "separate", idx.size)
    assert idx.size > 0
    old = oremap.layout(spec.oracle_plan, ocore.bf16(ph))
    want = oremap.remap(spec.oracle_plan, idx, val)
    pipe = _pipe(spec, n, old)
    tp, tm, tv = dev(p), dev(m), dev(v)
    if fused:
        pipe.step_fused(tp, tm, tv, hp)
    else:
        pipe.step(tp, tm, tv, hp)
    torch.cuda.synchronize()
    assert int(pipe.cursor.item()) == idx.size
    check_buckets(pipe, spec, want, old)
    pipe.close()
