"""Megatron-Core sender layout, on the CPU: pins of the oracle's converter
(appendix B, eq. mcore_fused_qkv, eq. mcore_tp_shard,
eq. canonical_qkv_unpacking) and of the product's plan composition.

Pins that do not lean on the oracle's own packing code:
  * hand-worked fused-QKV and fc1 row orders for tiny head counts;
  * the product plan of an MCore shard sends every element to exactly the
    receiver offsets that the torch-built dense receiver route of the
    canonical model holds for that element (tests/dense_route.py);
  * detection in the paper's order (inversion in MCore space, conversion,
    BF16 comparison in canonical space) equals detection on the canonical
    layout restricted to the sender rank's elements: the inversion and the
    BF16 cast are element-wise and conversion only moves elements.
"""
import numpy as np
import pytest
import torch

from oracle import mcore
from oracle import plan as oplan
from oracle import remap as oremap
from oracle import run as orun
from paper_2608_00455_amd import binding as B
from paper_2608_00455_amd import layouts
from synth import workloads as W

from dense_route import dense_receivers
from test_abi import _create_status

CASES = [
    lambda: W.scaled_mcore(),
    lambda: W.scaled_mcore(trainer_rank=1),
    lambda: W.scaled_mcore(trainer_tp=4, trainer_rank=2, receiver_tp=2),
    lambda: W.scaled_mcore(trainer_tp=2, trainer_rank=1, receiver_tp=4),
    lambda: W.scaled_mcore(layers=1, trainer_tp=1, receiver_tp=8, heads_q=8, heads_kv=8),
    lambda: W.scaled_mcore(layers=1, trainer_tp=2, trainer_rank=1, receiver_tp=4, vocab=96),
]


def test_fused_qkv_worked_example():
    # h_q = 4, h_kv = 2 (g = 2), d_h = 1, one input column: row labels
    # q0..q3 = 0..3, k0, k1 = 10, 11, v0, v1 = 20, 21.
    Wq = np.array([[0], [1], [2], [3]])
    Wk = np.array([[10], [11]])
    Wv = np.array([[20], [21]])
    fused = mcore.fuse_qkv(Wq, Wk, Wv, 4, 2, 1)
    assert fused[:, 0].tolist() == [0, 1, 10, 20, 2, 3, 11, 21]
    # TP = 2: rank 1 holds the second key/value group
    assert mcore.tp_shard(fused, 2, 1, 0)[:, 0].tolist() == [2, 3, 11, 21]
    q, k, v = mcore.unfuse_qkv(fused, 4, 2, 1)
    assert q[:, 0].tolist() == [0, 1, 2, 3] and k[:, 0].tolist() == [10, 11]
    assert v[:, 0].tolist() == [20, 21]


def test_fused_qkv_worked_example_two_rows_per_head():
    # h_q = 2, h_kv = 1 (g = 2), d_h = 2: [Q0; Q1; K0; V0] as 2-row blocks
    Wq = np.array([[0], [1], [2], [3]])
    Wk = np.array([[10], [11]])
    Wv = np.array([[20], [21]])
    assert mcore.fuse_qkv(Wq, Wk, Wv, 2, 1, 2)[:, 0].tolist() == [0, 1, 2, 3, 10, 11, 20, 21]


def test_fc1_worked_example():
    wl = W.scaled_mcore(layers=1, trainer_tp=2)
    u = [x for x in mcore.units(wl) if x.name.endswith("linear_fc1.weight")][0]
    gate = np.array([[0], [1], [2], [3]])
    up = np.array([[10], [11], [12], [13]])
    full = u.pack([gate, up])
    assert full[:, 0].tolist() == [0, 1, 10, 11, 2, 3, 12, 13]
    g2, u2 = u.unpack(full)
    assert g2[:, 0].tolist() == [0, 1, 2, 3] and u2[:, 0].tolist() == [10, 11, 12, 13]


@pytest.mark.parametrize("make", CASES)
def test_canonical_index_partitions_the_model(make):
    wl = make()
    P = wl.sender.tp
    n = W.canonical_twin(wl).numel
    count = np.zeros(n, np.int64)
    for r in range(P):
        ci = mcore.canonical_index(W.with_sender_rank(wl, r))
        assert np.unique(ci).size == ci.size
        count[ci] += 1
    replicated = np.zeros(n, bool)
    begins = wl.flat_begins()
    for k, t in enumerate(wl.tensors):
        if len(t.shape) == 1:
            replicated[begins[k]:begins[k] + t.numel] = True
    assert np.all(count[replicated] == P)
    assert np.all(count[~replicated] == 1)


@pytest.mark.parametrize("make", CASES)
def test_product_plan_routes_like_dense_receivers(make):
    wl = make()
    spec = layouts.build_spec(wl)
    assert _create_status(spec) in (B.DTE_OK, B.DTE_ERR_HIP)
    ci = mcore.canonical_index(wl)
    assert ci.size == spec.total
    ops = []
    for o in spec.c_ops():
        nd = len(spec.segments[o.segment][1])
        ops.append(oplan.Op(o.segment, o.rank, o.dst_base, tuple(o.src_origin[:nd]),
                            tuple(o.extent[:nd]), tuple(o.dst_origin[:nd]),
                            tuple(o.dst_shape[:nd])))
    pl = oplan.Plan([b for b, _ in spec.segments], [s for _, s in spec.segments], ops,
                    spec.rank_numel, [])
    got = oremap.remap(pl, np.arange(spec.total, dtype=np.int64), ci)
    twin = W.canonical_twin(wl)
    want = dense_receivers(twin, torch.arange(twin.numel))
    assert spec.rank_numel == [x.numel() for x in want]
    for r, (off, tag) in enumerate(got):
        w = want[r].numpy()
        assert np.array_equal(off, np.flatnonzero(np.isin(w, ci))), r
        assert np.array_equal(tag, w[off]), r


def test_canonical_sender_plan_unchanged():
    wl = W.scaled_dense(layers=2, tp=2)
    spec = layouts.build_spec(wl)
    assert [s.name for s in spec.senders] == [t.name for t in wl.tensors]


@pytest.mark.parametrize("make", CASES[:3])
def test_mcore_detection_equals_canonical_restricted(make):
    wl = make()
    hp = W.StepHP(lr=1e-5)
    got = mcore.extract(wl, hp)
    ref = orun.extract(W.canonical_twin(wl), hp=hp, threads=2)
    keep = np.isin(ref.idx, mcore.canonical_index(wl))
    assert got.idx.size > 0
    assert np.array_equal(got.idx, ref.idx[keep])
    assert np.array_equal(got.val, ref.val[keep])


def test_mcore_layout_rejects_moe_and_uneven_splits():
    with pytest.raises(ValueError):
        layouts.build_spec(W.scaled_mcore(trainer_tp=8))       # 4 kv heads over 8 ranks
