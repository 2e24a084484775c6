"""GPU parity of the Megatron-Core sender path (through the C ABI) against
the CPU oracle.

The product detects in the trainer rank's MCore layout and routes with a
plan whose operations carry the converter's permutation; the oracle follows
the paper's order (inversion in MCore space, gather and conversion to the
canonical tensors, BF16 comparison there, remap through the canonical plan).
Bit-exact: the delta (mapped to canonical offsets), the receiver buckets and
the applied receiver shards.
"""
import sys

import numpy as np
import pytest
import torch

import synth
from oracle import core as ocore
from oracle import mcore
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


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host_u16(t):
    return t.cpu().numpy().view(np.uint16)


def test_2d_device_draws_equal_host_draws():
    say("case: synth 2-D fill gpu vs cpu")
    rows, cols, stride = 333, 517, 601
    g = torch.full((rows * stride,), -3.0, dtype=torch.float32, device="cuda")
    for kind in range(4):
        synth.fill_gpu_2d(g.data_ptr(), rows, cols, stride, 777, 9, kind, 1000, 64, 2048)
        torch.cuda.synchronize()
        c = np.full((rows, stride), np.float32(-3.0))
        synth.fill_cpu_2d(c[:, :cols], 777, 9, kind, 1000, 64, 2048)
        assert np.array_equal(g.cpu().numpy().view(np.uint32), c.reshape(-1).view(np.uint32))


MCORE = [
    lambda: W.scaled_mcore(),
    lambda: W.scaled_mcore(trainer_rank=1),
    lambda: W.scaled_mcore(trainer_tp=4, trainer_rank=2, receiver_tp=2),
    lambda: W.scaled_mcore(layers=1, trainer_tp=2, trainer_rank=1, receiver_tp=4, vocab=96),
    lambda: W.scaled_mcore(layers=3, trainer_tp=2, trainer_rank=0, receiver_tp=8, hidden=256,
                           heads_q=16, heads_kv=8, head_dim=32, intermediate=704, vocab=512,
                           lr=1e-4),
    # norms in a parameter group without weight decay: one extract per run
    lambda: W.with_norm_group(W.scaled_mcore(trainer_rank=1, vocab=64, lr=1e-4)),
]


def check_mcore_path(wl, capacity_fraction=1.0):
    twin = W.canonical_twin(wl)
    ci = mcore.canonical_index(wl)
    want = mcore.extract(wl)
    say("  oracle: %d changes among %d sender elements" % (want.idx.size, ci.size))
    # receiver shards before the step: the canonical previous version everywhere
    res = orun.extract(twin, keep=("ph", "p"))
    cplan = oplan.build_plan(twin)
    old = oremap.layout(cplan, ocore.bf16(orun.flat(res.parts, "ph")))
    new_full = oremap.layout(cplan, ocore.bf16(orun.flat(res.parts, "p")))
    spec = layouts.build_spec(wl)
    assert spec.total == ci.size
    cap = max(1, int(ci.size * capacity_fraction))
    pipe = DeltaPipeline(spec, capacity=cap, shards=[dev(x.view(np.int16)) for x in old])
    p, m, v = generate_state(wl)
    assert p.numel() == ci.size
    pipe.step(p, m, v, wl.hp, runs=group_runs(wl))
    torch.cuda.synchronize()
    idx, val, total = pipe.delta()
    assert total == want.idx.size
    mapped = ci[idx]
    order = np.argsort(mapped, kind="stable")
    assert np.array_equal(mapped[order], want.idx)
    assert np.array_equal(val[order], want.val)
    buckets, counts = pipe.buckets()
    wb = oremap.remap(cplan, want.idx, want.val)
    expect = oremap.apply([x.copy() for x in old], wb)
    for r in range(cplan.nranks):
        assert counts[r] == wb[r][0].size, r
        assert np.array_equal(buckets[r][0], wb[r][0]), r
        assert np.array_equal(buckets[r][1], wb[r][1]), r
        got = host_u16(pipe.shards[r])
        assert np.array_equal(got, expect[r]), r
        # every element the sender rank holds now carries the current version
        held = np.zeros(cplan.rank_numel[r], bool)
        held[oremap.remap(cplan, ci, np.zeros(ci.size, np.uint16))[r][0]] = True
        assert np.array_equal(got[held], new_full[r][held]), r
    pipe.close()


@pytest.mark.parametrize("make", MCORE)
def test_mcore_full_path(make):
    wl = make()
    say("case: mcore full path", wl.name)
    check_mcore_path(wl)


def test_mcore_remap_of_every_offset():
    """Every MCore element changed: the plan sends each to the receiver
    offsets of its canonical element (tags = low 16 bits of the canonical
    offset)."""
    wl = W.scaled_mcore(trainer_tp=2, trainer_rank=1, receiver_tp=4)
    say("case: mcore remap all offsets", wl.name)
    ci = mcore.canonical_index(wl)
    n = ci.size
    tag = (ci * 2654435761 >> 7).astype(np.uint16)
    twin = W.canonical_twin(wl)
    cplan = oplan.build_plan(twin)
    want = oremap.remap(cplan, ci, tag)
    spec = layouts.build_spec(wl)
    pipe = DeltaPipeline(spec, capacity=n)
    pipe.idx.copy_(dev(np.arange(n, dtype=np.int64)))
    pipe.val.copy_(dev(tag.view(np.int16)))
    pipe.cursor.fill_(n)
    pipe.remap()
    torch.cuda.synchronize()
    buckets, counts = pipe.buckets()
    for r in range(cplan.nranks):
        assert counts[r] == want[r][0].size
        assert np.array_equal(buckets[r][0], want[r][0])
        assert np.array_equal(buckets[r][1], want[r][1])
    pipe.close()
