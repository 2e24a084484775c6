"""GPU side of the storage-mediated path (paper sec. 4.4): an ordered delta
published straight from the device and read back into device memory equals
the oracle's delta; remapped and applied on the GPU, it gives the receiver
layout of the new BF16 weights.  An unordered delta is refused."""
import sys

import numpy as np
import pytest
import torch

from oracle import core as ocore
from oracle import plan as oplan
from oracle import remap as oremap
from oracle import run as orun
from paper_2608_00455_amd import binding as B
from paper_2608_00455_amd import layouts
from paper_2608_00455_amd import store as S
from paper_2608_00455_amd.pipeline import DeltaPipeline, generate_state
from synth import workloads as W

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def segs_of(wl):
    return S.segments_of([t.name for t in wl.tensors], wl.flat_begins(),
                         [t.numel for t in wl.tensors])


@pytest.mark.parametrize("make,codec", [
    (lambda: W.scaled_dense(layers=2, tp=2, lr=1e-5), S.CODEC_ZSTD),
    (lambda: W.tiny_block(), S.CODEC_NONE),
    (lambda: W.tiny_block(), S.CODEC_ZSTD),
])
def test_publish_from_device_and_apply_on_device(tmp_path, make, codec):
    wl = make()
    say("case: store device round trip", wl.name, codec)
    res = orun.extract(wl, keep=("p", "m", "v", "ph"))
    st = {k: orun.flat(res.parts, k) for k in ("p", "m", "v", "ph")}
    p, m, v = dev(st["p"]), dev(st["m"]), dev(st["v"])
    spec = layouts.build_spec(wl)
    pipe = DeltaPipeline(spec, capacity=max(1, res.idx.size), ordered=True)
    pipe.reset()
    pipe.extract(p, m, v, wl.hp)
    d = tmp_path / "store"
    opt = S.Options(codec=codec, threads=4, chunk_entries=4096)
    stats = S.write_part_device(d, 1, 0, segs_of(wl), pipe.idx.data_ptr(), pipe.val.data_ptr(),
                                pipe.cursor.data_ptr(), pipe.capacity, opt,
                                torch.cuda.current_stream().cuda_stream)
    assert stats.entries == res.idx.size
    assert S.commit(d, 1, 0, 1)
    idx, val, _ = S.read_host(d, 1, 0)
    assert np.array_equal(idx, res.idx) and np.array_equal(val, res.val)
    # destination: read into device memory, remap and apply there
    pl = oplan.build_plan(wl)
    old = oremap.layout(pl, ocore.bf16(st["ph"]))
    new = oremap.layout(pl, ocore.bf16(st["p"]))
    dst = DeltaPipeline(spec, capacity=max(1, res.idx.size),
                        shards=[dev(x.view(np.int16)) for x in old])
    n, _ = S.read_device(d, 1, 0, dst.idx.data_ptr(), dst.val.data_ptr(), dst.capacity,
                         threads=4, stream=torch.cuda.current_stream().cuda_stream)
    assert n == res.idx.size
    dst.cursor.fill_(n)
    got_idx, got_val, _ = dst.delta(raw=True)
    assert np.array_equal(got_idx, res.idx) and np.array_equal(got_val, res.val)
    dst.remap()
    dst.apply()
    torch.cuda.synchronize()
    for r in range(pl.nranks):
        assert np.array_equal(dst.shards[r].cpu().numpy().view(np.uint16), new[r])
    pipe.close()
    dst.close()


def test_unordered_device_delta_is_refused(tmp_path):
    wl = W.scaled_dense(layers=1, tp=2, lr=1e-4)
    say("case: store refuses unordered delta")
    res = orun.extract(wl)
    idx = res.idx[::-1].copy()
    spec = layouts.build_spec(wl)
    pipe = DeltaPipeline(spec, capacity=idx.size)
    pipe.idx.copy_(dev(idx))
    pipe.val.copy_(dev(res.val[::-1].copy().view(np.int16)))
    pipe.cursor.fill_(idx.size)
    with pytest.raises(B.DteError) as e:
        S.write_part_device(tmp_path / "s", 1, 0, segs_of(wl), pipe.idx.data_ptr(),
                            pipe.val.data_ptr(), pipe.cursor.data_ptr(), pipe.capacity)
    assert e.value.status == B.DTE_ERR_ARG
    pipe.close()


def test_megatron_core_ranks_publish_from_device(tmp_path):
    """Two tensor-parallel Megatron-Core trainer ranks each extract their
    own shard (ordered) and publish it mapped to canonical tensors; the
    destination reads the version into device memory, remaps and applies
    it with the canonical model's receiver plan: the shards then hold the
    new BF16 weights everywhere."""
    wl0 = W.scaled_mcore(layers=2, trainer_tp=2, trainer_rank=0, receiver_tp=4, vocab=64,
                         lr=1e-5)
    twin = W.canonical_twin(wl0)
    say("case: store from mcore ranks", wl0.name)
    res = orun.extract(twin, keep=("ph", "p"))
    d = tmp_path / "store"
    segs = segs_of(twin)
    for r in range(2):
        wl = W.with_sender_rank(wl0, r)
        p, m, v = generate_state(wl)
        spec = layouts.build_spec(wl)
        pipe = DeltaPipeline(spec, capacity=p.numel(), ordered=True)
        pipe.reset()
        pipe.extract(p, m, v, wl.hp)
        S.write_part_device(d, 1, r, segs, pipe.idx.data_ptr(), pipe.val.data_ptr(),
                            pipe.cursor.data_ptr(), pipe.capacity, S.Options(chunk_entries=2000),
                            torch.cuda.current_stream().cuda_stream,
                            pieces=S.pieces_of(layouts.store_pieces(wl)))
        pipe.close()
    assert S.commit(d, 1, 0, 2)
    pl = oplan.build_plan(twin)
    old = oremap.layout(pl, ocore.bf16(orun.flat(res.parts, "ph")))
    new = oremap.layout(pl, ocore.bf16(orun.flat(res.parts, "p")))
    dst = DeltaPipeline(layouts.build_spec(twin), capacity=res.idx.size,
                        shards=[dev(x.view(np.int16)) for x in old])
    n, _ = S.read_device(d, 1, 0, dst.idx.data_ptr(), dst.val.data_ptr(), dst.capacity,
                         stream=torch.cuda.current_stream().cuda_stream)
    assert n == res.idx.size
    dst.cursor.fill_(n)
    idx, val, _ = dst.delta()
    assert np.array_equal(idx, res.idx) and np.array_equal(val, res.val)
    dst.remap()
    dst.apply()
    torch.cuda.synchronize()
    for r in range(pl.nranks):
        assert np.array_equal(dst.shards[r].cpu().numpy().view(np.uint16), new[r]), r
    dst.close()
