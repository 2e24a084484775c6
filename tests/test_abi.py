"""Host-side checks of the C ABI that need no GPU: every symbol declared in
include/dte.h is exported, scalar derivation matches the oracle bit for
bit, argument errors are reported before any device work, and plan
validation accepts the workload plans and rejects broken ones."""
import ctypes
import os
import re

import pytest

import synth
from oracle import core as ocore
from oracle import plan as oplan
from paper_2608_00455_amd import binding as B
from paper_2608_00455_amd import layouts
from synth import workloads as W

INCLUDE = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include")


def declared():
    names = set()
    for h in sorted(os.listdir(INCLUDE)):
        if h.endswith(".h"):
            text = open(os.path.join(INCLUDE, h)).read()
            names |= set(re.findall(r"^[A-Za-z_][\w \t\*]*?\b(dte_\w+)\s*\(", text, re.M))
    return sorted(names)


def test_every_declared_symbol_is_exported():
    from paper_2608_00455_amd import store
    names = declared()
    assert set(names) == set(B.EXPORTED) | set(store.EXPORTED)
    lib = ctypes.CDLL(B.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


@pytest.mark.parametrize("lr", [0.0, 1e-7, 1e-6, 1e-5, 1e-4, 3e-3])
@pytest.mark.parametrize("step", [1, 7, 100, 5000])
@pytest.mark.parametrize("wd", [0.0, 0.01, 0.1])
@pytest.mark.parametrize("order", [W.ORDER_FOLDED, W.ORDER_LITERAL])
def test_scalars_bit_equal_oracle(lr, step, wd, order):
    hp = W.StepHP(lr=lr, step=step, weight_decay=wd, order=order)
    got = B.dte_derive_scalars(hp)
    want = ocore.derive_scalars(hp)
    for f in ("lrb1", "rbc2", "eps", "decay", "lr", "bc1", "bc2"):
        a = ctypes.c_float(getattr(got, f))
        b = ctypes.c_float(getattr(want, f))
        assert bytes(a) == bytes(b), f
    assert got.order == want.order == order


@pytest.mark.parametrize("bad", [
    dict(step=0), dict(beta1=1.0), dict(beta2=-0.1), dict(lr=-1e-6), dict(lr=float("nan")),
    dict(lr=100.0, weight_decay=0.01), dict(eps=float("inf")), dict(order=2), dict(reserved=1),
])
def test_invalid_hyperparameters(bad):
    hp = B.dte_adamw_step(1e-6, 0.9, 0.999, 1e-8, 0.01, 100)
    for k, v in bad.items():
        setattr(hp, k, v)
    st = B.raw_status("dte_derive_scalars", ctypes.byref(hp), ctypes.byref(B.dte_scalars()))
    assert st == B.DTE_ERR_ARG
    st = B.raw_status("dte_extract_delta", 16, 16, 16, 4, 0, ctypes.byref(hp), 16, 16, 4, 16,
                      None, None)
    assert st == B.DTE_ERR_ARG


def test_argument_errors_and_empty_calls():
    hp = B.dte_adamw_step(1e-6, 0.9, 0.999, 1e-8, 0.01, 100)
    ext = lambda *a: B.raw_status("dte_extract_delta", *a)  # noqa: E731
    assert ext(16, 16, 16, -1, 0, ctypes.byref(hp), 16, 16, 4, 16, None, None) == B.DTE_ERR_ARG
    assert ext(16, 16, 16, 4, -5, ctypes.byref(hp), 16, 16, 4, 16, None, None) == B.DTE_ERR_ARG
    assert ext(None, 16, 16, 4, 0, ctypes.byref(hp), 16, 16, 4, 16, None, None) == B.DTE_ERR_ARG
    assert ext(16, 16, 16, 4, 0, ctypes.byref(hp), None, 16, 4, 16, None, None) == B.DTE_ERR_ARG
    assert ext(16, 16, 16, 4, 0, ctypes.byref(hp), 16, 16, -1, 16, None, None) == B.DTE_ERR_ARG
    assert ext(16, 16, 16, 4, 0, ctypes.byref(hp), 16, 16, 4, None, None, None) == B.DTE_ERR_ARG
    assert ext(16, 16, 16, 4, 0, None, 16, 16, 4, 16, None, None) == B.DTE_ERR_ARG
    # zero-length input: legal, nothing enqueued (no device needed)
    assert ext(None, None, None, 0, 0, ctypes.byref(hp), None, None, 0, None, None,
               None) == B.DTE_OK
    fwd = lambda *a: B.raw_status("dte_adamw_forward", *a)  # noqa: E731
    assert fwd(None, None, None, None, 0, ctypes.byref(hp), None) == B.DTE_OK
    assert fwd(16, 16, None, 16, 4, ctypes.byref(hp), None) == B.DTE_ERR_ARG
    assert B.raw_status("dte_plan_info", None, None, None, None) == B.DTE_ERR_ARG
    assert B.raw_status("dte_remap", None, 16, 16, 16, 4, None, None, None, 16,
                        None) == B.DTE_ERR_ARG
    assert B.raw_status("dte_apply", None, None, None, None, 16, None, None) == B.DTE_ERR_ARG
    B.dte_plan_destroy(None)
    assert "ERR_PLAN" in B.dte_status_string(B.DTE_ERR_PLAN)


def test_noalloc_capacity_limit():
    """The no-allocation ordered call takes capacities whose workspace fits
    its 64 MiB static array and rejects larger ones before any device work."""
    cap = B.dte_ordered_noalloc_max_capacity()
    assert B.dte_ordered_workspace_bytes(cap) <= 64 << 20 < B.dte_ordered_workspace_bytes(cap + 1)
    assert cap > 3_000_000
    hp = B.dte_adamw_step(1e-6, 0.9, 0.999, 1e-8, 0.01, 100)
    call = lambda *a: B.raw_status("dte_extract_delta_ordered_noalloc", *a)  # noqa: E731
    assert call(16, 16, 16, 4, 0, ctypes.byref(hp), 16, 16, cap + 1, 16, None,
                None) == B.DTE_ERR_CAPACITY
    assert call(16, 16, 16, -1, 0, ctypes.byref(hp), 16, 16, 4, 16, None, None) == B.DTE_ERR_ARG
    assert call(None, None, None, 0, 0, ctypes.byref(hp), None, None, 0, None, None,
                None) == B.DTE_OK


def test_every_status_code_has_its_own_name():
    codes = [B.DTE_OK, B.DTE_ERR_ARG, B.DTE_ERR_PLAN, B.DTE_ERR_CAPACITY, B.DTE_ERR_HIP,
             B.DTE_ERR_IO, B.DTE_ERR_CORRUPT, B.DTE_ERR_CHAIN, B.DTE_ERR_UNSUPPORTED,
             B.DTE_ERR_HOST]
    assert codes == list(range(10))
    names = [B.dte_status_string(c) for c in codes]
    assert len(set(names)) == len(names)
    assert names[0] == "DTE_OK" and names[9].startswith("DTE_ERR_HOST")
    assert B.dte_status_string(10) == "unknown dte_status"


def _create_status(spec, segs=None, ops=None, numel=None):
    segs = segs if segs is not None else spec.c_segments()
    ops = ops if ops is not None else spec.c_ops()
    numel = numel if numel is not None else spec.rank_numel
    sa = (B.dte_segment * len(segs))(*segs)
    oa = (B.dte_op * max(1, len(ops)))(*ops)
    na = (ctypes.c_int64 * len(numel))(*numel)
    h = ctypes.c_void_p()
    st = B.raw_status("dte_plan_create", sa, len(segs), oa, len(ops), len(numel), na,
                      ctypes.byref(h))
    if st == B.DTE_OK:
        B.dte_plan_destroy(h.value)
    return st


WORKLOADS = [
    lambda: W.tiny_block(),
    lambda: W.scaled_dense(layers=2, tp=2),
    lambda: W.scaled_moe(synth.word, layers=2, ranks=4, attn_tp=2, experts=8),
    lambda: W.qwen3_8b(4),
    lambda: W.qwen3_8b(8),
    lambda: W.qwen3_30b_a3b_share(synth.word),
    lambda: W.qwen3_8b_layers_sweep(1e-6),
]


@pytest.mark.parametrize("make", WORKLOADS)
def test_workload_plans_pass_validation(make):
    spec = layouts.build_spec(make())
    # without a GPU the upload fails after validation (DTE_ERR_HIP)
    assert _create_status(spec) in (B.DTE_OK, B.DTE_ERR_HIP)


@pytest.mark.parametrize("make", WORKLOADS)
def test_product_plan_equals_oracle_plan(make):
    wl = make()
    spec = layouts.build_spec(wl)
    pl = oplan.build_plan(wl)
    assert spec.rank_numel == pl.rank_numel
    assert [s for _, s in spec.segments] == pl.seg_shape
    assert [b for b, _ in spec.segments] == pl.seg_begin

    def key_c(o, nd):
        return (o.segment, o.rank, o.dst_base, tuple(o.src_origin[:nd]), tuple(o.extent[:nd]),
                tuple(o.dst_origin[:nd]), tuple(o.dst_shape[:nd]))

    mine = sorted(key_c(o, len(spec.segments[o.segment][1])) for o in spec.c_ops())
    theirs = sorted((o.segment, o.rank, o.dst_base, o.src_origin, o.extent, o.dst_origin,
                     o.dst_shape) for o in pl.ops)
    assert mine == theirs


def _tiny_spec():
    return layouts.build_spec(W.scaled_dense(layers=1, tp=2))


def test_plan_rejects_overlapping_destinations():
    spec = _tiny_spec()
    ops = spec.c_ops()
    ops[1].dst_base = ops[0].dst_base          # second view lands on the first
    ops[1].dst_shape[:] = ops[0].dst_shape[:]
    assert _create_status(spec, ops=ops) == B.DTE_ERR_PLAN


def test_plan_rejects_uncovered_segment():
    spec = _tiny_spec()
    ops = [o for o in spec.c_ops() if not (o.segment == 1 and o.rank == 1)]
    assert _create_status(spec, ops=ops) == B.DTE_ERR_PLAN


def test_plan_rejects_out_of_bounds():
    spec = _tiny_spec()
    ops = spec.c_ops()
    ops[3].dst_base = spec.rank_numel[ops[3].rank]     # view past the end of the rank
    assert _create_status(spec, ops=ops) == B.DTE_ERR_PLAN
    ops = spec.c_ops()
    ops[2].extent[0] += 1                               # box past the segment
    assert _create_status(spec, ops=ops) == B.DTE_ERR_PLAN
    ops = spec.c_ops()
    ops[0].rank = 7                                     # unknown rank
    assert _create_status(spec, ops=ops) == B.DTE_ERR_PLAN


def test_plan_rejects_bad_segments():
    spec = _tiny_spec()
    segs = spec.c_segments()
    segs[2].flat_begin += 1                             # gap between segments
    assert _create_status(spec, segs=segs) == B.DTE_ERR_PLAN
    segs = spec.c_segments()
    segs[0].ndim = 5
    assert _create_status(spec, segs=segs) == B.DTE_ERR_PLAN


def test_plan_rejects_duplicate_source_for_one_rank():
    spec = _tiny_spec()
    ops = spec.c_ops()
    dup = B.dte_op.from_buffer_copy(ops[0])
    # same source box to the same rank, into a fresh view past the old end
    numel = list(spec.rank_numel)
    nd = len(spec.segments[dup.segment][1])
    size = 1
    for d in range(nd):
        size *= dup.dst_shape[d]
    dup.dst_base = numel[dup.rank]
    numel[dup.rank] += size
    assert _create_status(spec, ops=ops + [dup], numel=numel) == B.DTE_ERR_PLAN


def test_ordered_workspace_and_argument_errors():
    assert B.dte_ordered_workspace_bytes(-1) == -1
    assert B.dte_ordered_workspace_bytes(1 << 41) == -1
    small = B.dte_ordered_workspace_bytes(0)
    big = B.dte_ordered_workspace_bytes(1_000_000)
    assert small > 0 and small % 256 == 0
    assert big >= small + 20 * 1_000_000
    hp = B.dte_adamw_step(1e-6, 0.9, 0.999, 1e-8, 0.01, 100)
    ext = lambda *a: B.raw_status("dte_extract_delta_ordered", *a)  # noqa: E731
    need = B.dte_ordered_workspace_bytes(4)
    # zero-length input: legal, nothing enqueued
    assert ext(None, None, None, 0, 0, ctypes.byref(hp), None, None, 0, None, None, 0, None,
               None) == B.DTE_OK
    # missing, too small or misaligned workspace
    assert ext(16, 16, 16, 4, 0, ctypes.byref(hp), 16, 16, 4, 16, None, need, None,
               None) == B.DTE_ERR_ARG
    assert ext(16, 16, 16, 4, 0, ctypes.byref(hp), 16, 16, 4, 16, 256, need - 1, None,
               None) == B.DTE_ERR_ARG
    assert ext(16, 16, 16, 4, 0, ctypes.byref(hp), 16, 16, 4, 16, 16, need, None,
               None) == B.DTE_ERR_ARG
    assert ext(16, 16, 16, -1, 0, ctypes.byref(hp), 16, 16, 4, 16, 256, need, None,
               None) == B.DTE_ERR_ARG


def test_high_dimensional_plan_passes_validation():
    from highdim_plan import HighDimSpec
    spec = HighDimSpec()
    assert _create_status(spec) in (B.DTE_OK, B.DTE_ERR_HIP)
