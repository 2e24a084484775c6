"""GPU parity with two parameter groups (norms without weight decay,
sec. 4.1): the state is generated and the delta extracted per run of
segments with equal step scalars, appending to one delta; compared bit for
bit with the oracle, including the reconstructed weights."""
import sys

import numpy as np
import pytest
import torch

from oracle import core as ocore
from oracle import plan as oplan
from oracle import remap as oremap
from oracle import run as orun
from paper_2608_00455_amd import layouts
from paper_2608_00455_amd.pipeline import DeltaPipeline, generate_state, group_runs
from synth import workloads as W

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("lr", [1e-6, 1e-5, 1e-4])
def test_grouped_full_path_small_dense(lr):
    wl = W.with_norm_group(W.scaled_dense(layers=2, tp=2, lr=lr))
    say("case: parameter groups", wl.name, lr)
    res = orun.extract(wl, keep=("ph", "p"))
    pl = oplan.build_plan(wl)
    old = oremap.layout(pl, ocore.bf16(orun.flat(res.parts, "ph")))
    new = oremap.layout(pl, ocore.bf16(orun.flat(res.parts, "p")))
    spec = layouts.build_spec(wl)
    runs = group_runs(wl)
    assert len(runs) == (1 if lr < 3e-6 else 9)
    p, m, v = generate_state(wl)
    assert np.array_equal(p.cpu().numpy().view(np.uint32),
                          orun.flat(res.parts, "p").view(np.uint32))
    shards = [torch.from_numpy(x.view(np.int16)).cuda() for x in old]
    pipe = DeltaPipeline(spec, capacity=wl.numel, shards=shards)
    pipe.step(p, m, v, wl.hp, runs=runs)
    torch.cuda.synchronize()
    idx, val, total = pipe.delta()
    assert total == res.idx.size
    assert np.array_equal(idx, res.idx) and np.array_equal(val, res.val)
    buckets, counts = pipe.buckets()
    want = oremap.remap(pl, res.idx, res.val)
    for r in range(pl.nranks):
        assert np.array_equal(buckets[r][0], want[r][0])
        assert np.array_equal(buckets[r][1], want[r][1])
        assert np.array_equal(pipe.shards[r].cpu().numpy().view(np.uint16), new[r])
    # reconstructed weights of every group, 0 ulp
    prev = torch.empty_like(p)
    pipe.reset()
    pipe.extract_runs(p, m, v, runs, out_prev=prev)
    torch.cuda.synchronize()
    assert np.array_equal(prev.cpu().numpy().view(np.uint32),
                          orun.flat(res.parts, "ph").view(np.uint32))
    pipe.close()
