"""Pins of the oracle's detection/compaction (sec. 4.2.1) and direct sparse
apply (sec. 4.3): brute force on small inputs and the invariants of
sending target values (idempotent apply, untouched elements kept,
apply(layout(old), delta) == layout(new))."""
import numpy as np
import pytest

from oracle import core
from oracle import plan as oplan
from oracle import remap as oremap
from oracle import run as orun
from synth import workloads as W


def test_detect_equals_bruteforce_loop():
    wl = W.scaled_dense(layers=1, tp=2, lr=1e-4)
    res = orun.extract(wl, keep=("ph", "p"), threads=1)
    ph = orun.flat(res.parts, "ph")
    p = orun.flat(res.parts, "p")
    idx, val = [], []
    for i in range(p.size):                     # one element at a time
        a = core.lib().oracle_bf16(float(ph[i]))
        b = core.lib().oracle_bf16(float(p[i]))
        if a != b:
            idx.append(i)
            val.append(b)
    assert len(idx) > 100
    assert np.array_equal(res.idx, np.array(idx, np.int64))
    assert np.array_equal(res.val, np.array(val, np.uint16))
    assert np.all(np.diff(res.idx) > 0)          # ascending, unique


@pytest.fixture(scope="module")
def tiny():
    wl = W.tiny_block()
    res = orun.extract(wl, keep=("ph", "p", "p_prev"))
    pl = oplan.build_plan(wl)
    return wl, res, pl


def test_apply_invariant_and_idempotence(tiny):
    wl, res, pl = tiny
    ph, p = orun.flat(res.parts, "ph"), orun.flat(res.parts, "p")
    old = oremap.layout(pl, core.bf16(ph))
    new = oremap.layout(pl, core.bf16(p))
    buckets = oremap.remap(pl, res.idx, res.val)
    once = oremap.apply([s.copy() for s in old], buckets)
    for r in range(pl.nranks):
        assert np.array_equal(once[r], new[r])
    twice = oremap.apply([s.copy() for s in once], buckets)
    for r in range(pl.nranks):
        assert np.array_equal(twice[r], once[r])
    # elements outside the payload are untouched
    for r, (off, _) in enumerate(buckets):
        keep = np.ones(pl.rank_numel[r], bool)
        keep[off] = False
        assert np.array_equal(once[r][keep], old[r][keep])
    assert res.diag.changed == res.idx.size > 0


def test_apply_against_true_previous_weights(tiny):
    """With old := layout(b(p_prev)) the result differs from layout(b(p))
    exactly where b(p_prev) != b(ph) and b(ph) == b(p)."""
    wl, res, pl = tiny
    ph, p, pp = (orun.flat(res.parts, x) for x in ("ph", "p", "p_prev"))
    b_prev, b_ph, b_p = core.bf16(pp), core.bf16(ph), core.bf16(p)
    old = oremap.layout(pl, b_prev)
    new = oremap.layout(pl, b_p)
    got = oremap.apply([s.copy() for s in old], oremap.remap(pl, res.idx, res.val))
    missed = np.flatnonzero((b_prev != b_ph) & (b_ph == b_p))
    assert missed.size == res.diag.apply_vs_prev_diff
    # replication of each missed element = number of receivers holding it
    want = sum(b[0].size for b in oremap.remap(pl, missed, b_p[missed]))
    assert sum(int(np.count_nonzero(got[r] != new[r])) for r in range(pl.nranks)) == want


def test_lr_zero_gives_empty_delta():
    wl = W.scaled_dense(layers=1, tp=2)
    res = orun.extract(wl, hp=W.StepHP(lr=0.0), threads=1)
    assert res.idx.size == 0 and res.diag.fp32_recon_mismatch == 0


def test_tiny_block_diagnostics_match_golden():
    """Regression pin of the oracle's counts (tests/golden/diagnostics.json,
    written by python -m oracle.diagnostics)."""
    import json
    import os
    gold = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                       "diagnostics.json")))["workloads"]["tiny_block_tp2"]
    d = orun.extract(W.tiny_block()).diag
    assert (d.n, d.changed, d.bf16_recon_mismatch, d.fp32_recon_mismatch, d.true_changed,
            d.apply_vs_prev_diff) == (gold["elements"], gold["changed"],
                                      gold["bf16_recon_mismatch"], gold["fp32_recon_mismatch"],
                                      gold["true_changed"], gold["apply_vs_prev_diff"])
