"""GPU parity of the HIP path (through the C ABI) against the CPU oracle.

Bit-exact: delta index set, BF16 values, reconstructed binary32 weights
(0 ulp), remapped (rank, offset, value) entries and applied shards; the
capacity / count semantics; edge cases (empty, ragged, misaligned,
special values, DECAY != 1, many ranks).
"""
import sys

import numpy as np
import pytest
import torch

import synth
from oracle import core as ocore
from oracle import plan as oplan
from oracle import remap as oremap
from oracle import run as orun
from paper_2608_00455_amd import binding as B
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


def sync():
    torch.cuda.synchronize()


def oracle_state(wl, hp=None):
    res = orun.extract(wl, hp=hp, keep=("p", "m", "v", "ph", "p_prev"))
    return res, {k: orun.flat(res.parts, k) for k in ("p", "m", "v", "ph", "p_prev")}


def assert_delta_equal(pipe, res):
    idx, val, total = pipe.delta()
    assert total == res.idx.size
    assert np.array_equal(idx, res.idx)
    assert np.array_equal(val, res.val)


def test_synth_device_draws_equal_host_draws():
    say("case: synth fill gpu vs cpu")
    n = 1_000_003
    for kind in range(4):
        g = torch.empty(n, dtype=torch.float32, device="cuda")
        synth.fill_gpu(g.data_ptr(), n, 4242, 17, kind, 123_456_789)
        sync()
        c = synth.draw_cpu(n, 4242, 17, kind, 123_456_789)
        assert np.array_equal(g.cpu().numpy().view(np.uint32), c.view(np.uint32)), kind


def test_forward_step_equals_oracle():
    wl = W.scaled_moe(synth.word, layers=1, ranks=4, attn_tp=2, experts=8)
    say("case: adamw forward", wl.name)
    p, m, v = generate_state(wl)
    _, st = oracle_state(wl)
    for name, t in (("p", p), ("m", m), ("v", v)):
        assert np.array_equal(t.cpu().numpy().view(np.uint32), st[name].view(np.uint32)), name


@pytest.fixture(scope="module")
def tiny():
    wl = W.tiny_block()
    res, st = oracle_state(wl)
    return wl, res, st


def test_extract_on_oracle_inputs_tiny_block(tiny):
    wl, res, st = tiny
    say("case: extract tiny_block on oracle inputs")
    spec = layouts.build_spec(wl)
    pipe = DeltaPipeline(spec, capacity=wl.numel)
    p, m, v = dev(st["p"]), dev(st["m"]), dev(st["v"])
    prev = torch.empty_like(p)
    pipe.reset()
    pipe.extract(p, m, v, wl.hp, out_prev=prev)
    sync()
    assert_delta_equal(pipe, res)
    assert np.array_equal(prev.cpu().numpy().view(np.uint32), st["ph"].view(np.uint32))
    pipe.close()


def test_full_path_tiny_block_generated_state(tiny):
    wl, res, st = tiny
    say("case: full path tiny_block, device-generated state")
    p, m, v = generate_state(wl)
    pl = oplan.build_plan(wl)
    old = oremap.layout(pl, ocore.bf16(st["ph"]))
    new = oremap.layout(pl, ocore.bf16(st["p"]))
    spec = layouts.build_spec(wl)
    pipe = DeltaPipeline(spec, capacity=wl.numel // 16, shards=[dev(x.view(np.int16)) for x in old])
    pipe.step(p, m, v, wl.hp)
    sync()
    assert_delta_equal(pipe, res)
    buckets, counts = pipe.buckets()
    want = oremap.remap(pl, res.idx, res.val)
    for r in range(pl.nranks):
        assert counts[r] == want[r][0].size
        assert np.array_equal(buckets[r][0], want[r][0])
        assert np.array_equal(buckets[r][1], want[r][1])
    for r in range(pl.nranks):
        assert np.array_equal(host_u16(pipe.shards[r]), new[r]), r
    # applying the same delta again changes nothing (target values)
    pipe.apply()
    sync()
    for r in range(pl.nranks):
        assert np.array_equal(host_u16(pipe.shards[r]), new[r]), r
    pipe.close()


@pytest.mark.parametrize("order", [W.ORDER_FOLDED, W.ORDER_LITERAL])
@pytest.mark.parametrize("lr", [0.0, 1e-7, 1e-6, 1e-5, 1e-4, 1e-2])
def test_learning_rates_small_dense(lr, order):
    wl = W.scaled_dense(layers=2, tp=2, lr=lr)
    hp = W.StepHP(lr=lr, order=order)
    say("case: lr sweep", wl.name, lr, order)
    res, st = oracle_state(wl, hp)
    spec = layouts.build_spec(wl)
    pipe = DeltaPipeline(spec, capacity=wl.numel)
    # the device forward step in the same order gives the same state
    gp, gm, gv = generate_state(wl, hp)
    for name, t in (("p", gp), ("m", gm), ("v", gv)):
        assert np.array_equal(t.cpu().numpy().view(np.uint32), st[name].view(np.uint32)), name
    del gp, gm, gv
    p, m, v = dev(st["p"]), dev(st["m"]), dev(st["v"])
    prev = torch.empty_like(p)
    pipe.reset()
    pipe.extract(p, m, v, hp, out_prev=prev)
    pipe.remap()
    sync()
    assert_delta_equal(pipe, res)
    assert np.array_equal(prev.cpu().numpy().view(np.uint32), st["ph"].view(np.uint32))
    buckets, counts = pipe.buckets()
    want = oremap.remap(oplan.build_plan(wl), res.idx, res.val)
    for r in range(len(want)):
        assert np.array_equal(buckets[r][0], want[r][0])
        assert np.array_equal(buckets[r][1], want[r][1])
    if lr == 0.0:
        assert res.idx.size == 0
    # the filtered path (no theta_hat requested) finds the same delta
    pipe.reset()
    pipe.extract(p, m, v, hp)
    sync()
    assert_delta_equal(pipe, res)
    pipe.close()


def test_ragged_misaligned_and_appended_ranges():
    wl = W.scaled_dense(layers=1, tp=2, lr=1e-4)
    say("case: ragged / misaligned / append")
    res, st = oracle_state(wl)
    n = 4096 * 3 + 13
    p, m, v = (st[k][:n] for k in ("p", "m", "v"))
    want_idx, want_val, want_ph = ocore.detect(p, m, v, ocore.derive_scalars(wl.hp), 0)
    spec = layouts.build_spec(wl)
    pipe = DeltaPipeline(spec, capacity=n)
    P, M, V = dev(p), dev(m), dev(v)
    prev = torch.zeros(n + 1, dtype=torch.float32, device="cuda")
    for cut in (0, 1, 4095, 4097, 6001, n - 1, n):
        pipe.reset()
        # [0, cut) from aligned bases; [cut, n) from bases offset by `cut`
        # elements (odd cut: misaligned, scalar-load path)
        pipe.extract(P, M, V, wl.hp, n=cut, index_base=0, out_prev=prev)
        pipe.extract(P[cut:], M[cut:], V[cut:], wl.hp, n=n - cut, index_base=cut,
                     out_prev=prev[cut:])
        sync()
        idx, val, total = pipe.delta()
        assert total == want_idx.size, cut
        assert np.array_equal(idx, want_idx) and np.array_equal(val, want_val), cut
        assert np.array_equal(prev[:n].cpu().numpy().view(np.uint32), want_ph.view(np.uint32))
    # ragged length on aligned buffers (vector path with a partial last tile)
    for m_len in (1, 3, 4, 5, 4096, 4099, 8191):
        pipe.reset()
        pipe.extract(P, M, V, wl.hp, n=m_len)
        sync()
        idx, val, total = pipe.delta()
        sel = want_idx < m_len
        assert np.array_equal(idx, want_idx[sel]) and np.array_equal(val, want_val[sel]), m_len
    pipe.close()


@pytest.mark.parametrize("base", [1000, (1 << 40) + 7])
@pytest.mark.parametrize("order", [W.ORDER_FOLDED, W.ORDER_LITERAL])
def test_special_values(order, base):
    """index_base 2^40 + 7: offsets far beyond 32 bits come out exact."""
    say("case: special values", order, base)
    rng = np.random.default_rng(3)
    n = 5000
    p = (rng.standard_normal(n) * 0.02).astype(np.float32)
    m = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    v = np.abs(rng.standard_normal(n) * 1e-6).astype(np.float32)
    specials = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, 1e-45, -1e-45, 1e-40, 3e38,
                         -3e38, 1.0, -1.0, 65504.0, 1.17549435e-38], np.float32)
    k = specials.size
    for j in range(0, 600, k):
        p[j:j + k] = specials
        m[j + 200:j + 200 + k] = specials
        v[j + 400:j + 400 + k] = specials
    p[4000:4010] = np.array([0x3F808000, 0x3F807FFF, 0x3F818000, 0x7F7F8000, 0x00008000,
                             0x80000001, 0x7F800001, 0xFFC00000, 0x007F8000, 0x3FFF8000],
                            np.uint32).view(np.float32)
    for lr in (1e-6, 1e-4, 3e-1):
        hp = W.StepHP(lr=lr, order=order)
        sc = ocore.derive_scalars(hp)
        want_idx, want_val, want_ph = ocore.detect(p, m, v, sc, base)
        spec = layouts.build_spec(W.scaled_dense(layers=1, tp=2))
        pipe = DeltaPipeline(spec, capacity=n)
        prev = torch.empty(n, dtype=torch.float32, device="cuda")
        pipe.reset()
        pipe.extract(dev(p), dev(m), dev(v), hp, index_base=base, out_prev=prev)
        sync()
        idx, val, total = pipe.delta()
        assert np.array_equal(idx, want_idx) and np.array_equal(val, want_val), lr
        got_ph = prev.cpu().numpy()
        nan = np.isnan(want_ph)
        assert np.array_equal(np.isnan(got_ph), nan)
        assert np.array_equal(got_ph.view(np.uint32)[~nan], want_ph.view(np.uint32)[~nan])
        # and through the "unchanged" proof (no theta_hat requested)
        pipe.reset()
        pipe.extract(dev(p), dev(m), dev(v), hp, index_base=base)
        sync()
        idx, val, total = pipe.delta()
        assert np.array_equal(idx, want_idx) and np.array_equal(val, want_val), lr
        pipe.close()


def test_capacity_overflow_reports_true_total(tiny):
    wl, res, st = tiny
    say("case: capacity overflow")
    spec = layouts.build_spec(wl)
    cap = res.idx.size // 3
    pipe = DeltaPipeline(spec, capacity=cap, rank_capacity=[cap // 2, 7])
    pipe.step(dev(st["p"]), dev(st["m"]), dev(st["v"]), wl.hp)
    sync()
    idx, val, total = pipe.delta()
    assert total == res.idx.size and idx.size == cap
    assert np.unique(idx).size == cap
    pos = np.searchsorted(res.idx, idx)
    assert np.array_equal(res.idx[pos], idx) and np.array_equal(res.val[pos], val)
    # buckets: a duplicate-free subset of the oracle's buckets of the full
    # delta, truncated at each rank's capacity
    buckets, counts = pipe.buckets()
    full = oremap.remap(oplan.build_plan(wl), res.idx, res.val)
    for r in range(2):
        got_off, got_val = buckets[r]
        assert got_off.size == min(counts[r], pipe.rank_capacity[r])
        assert counts[r] <= full[r][0].size
        assert np.unique(got_off).size == got_off.size
        pos = np.searchsorted(full[r][0], got_off)
        assert np.array_equal(full[r][0][pos], got_off)
        assert np.array_equal(full[r][1][pos], got_val)
    pipe.close()


@pytest.mark.parametrize("make", [
    lambda: W.tiny_block(),
    lambda: W.scaled_moe(synth.word, layers=2, ranks=8, attn_tp=2, experts=16, hidden=64,
                         head_dim=16, expert_intermediate=24),
    lambda: W.scaled_dense(layers=1, tp=32, heads_q=32, heads_kv=32, head_dim=8, hidden=64,
                           intermediate=128, vocab=64),
])
def test_remap_and_apply_of_every_offset(make):
    """Remap of idx = arange(N) (every element changed) against the oracle:
    a bijection onto the receiver shards; apply fills every element."""
    wl = make()
    say("case: remap all offsets", wl.name)
    n = wl.numel
    pl = oplan.build_plan(wl)
    idx = np.arange(n, dtype=np.int64)
    val = (idx * 2654435761 >> 7).astype(np.uint16)
    want = oremap.remap(pl, idx, val)
    spec = layouts.build_spec(wl)
    pipe = DeltaPipeline(spec, capacity=n)
    pipe.idx.copy_(dev(idx))
    pipe.val.copy_(dev(val.view(np.int16)))
    pipe.cursor.fill_(n)
    pipe.remap()
    pipe.apply()
    sync()
    buckets, counts = pipe.buckets()
    for r in range(pl.nranks):
        assert counts[r] == pl.rank_numel[r]
        assert np.array_equal(buckets[r][0], np.arange(pl.rank_numel[r]))
        assert np.array_equal(buckets[r][1], want[r][1])
        assert np.array_equal(host_u16(pipe.shards[r]), want[r][1])
    pipe.close()


def test_empty_delta_leaves_shards_untouched():
    wl = W.scaled_dense(layers=1, tp=2, lr=0.0)
    say("case: empty delta")
    spec = layouts.build_spec(wl)
    sentinel = [torch.full((n,), 0x7FFF, dtype=torch.int16, device="cuda")
                for n in spec.rank_numel]
    pipe = DeltaPipeline(spec, capacity=1024, shards=sentinel)
    p, m, v = generate_state(wl)
    pipe.step(p, m, v, wl.hp)
    sync()
    assert pipe.delta()[2] == 0
    assert int(pipe.rank_count.sum().item()) == 0
    for s in pipe.shards:
        assert bool((s == 0x7FFF).all())
    pipe.close()


@pytest.mark.parametrize("lr", [1e-7, 1e-6, 1e-4, 3e-2])
@pytest.mark.parametrize("order", [W.ORDER_FOLDED, W.ORDER_LITERAL])
def test_values_at_bf16_rounding_midpoints(lr, order):
    """Weights a few binary32 ulps from BF16 rounding midpoints (where the
    reconstruction decides the pattern), zeros, subnormals and both signs of
    the moment: every element parity-checked against the oracle."""
    say("case: rounding midpoints", lr)
    rng = np.random.default_rng(11)
    n = 1 << 18
    hi = rng.integers(0, 1 << 16, n, dtype=np.uint32)
    hi = (hi & 0x80FF) | (rng.integers(0x30, 0x42, n, dtype=np.uint32) << 7)  # |p| ~ 1e-7..8
    low = (0x8000 + rng.integers(-40, 41, n)).astype(np.uint32) & 0xFFFF
    pbits = (hi << 16) | low
    pbits[:64] = np.arange(64, dtype=np.uint32)                 # +0 and subnormals
    pbits[64:128] = np.arange(64, dtype=np.uint32) | 0x80000000  # -0 and negative subnormals
    p = pbits.view(np.float32)
    m = (rng.standard_normal(n) * 10.0 ** rng.uniform(-9, -2, n)).astype(np.float32)
    m[::7] = 0.0
    m[1::7] = -0.0
    v = np.abs(rng.standard_normal(n) * 10.0 ** rng.uniform(-12, -4, n)).astype(np.float32)
    v[::5] = 0.0
    hp = W.StepHP(lr=lr, order=order)
    want_idx, want_val, _ = ocore.detect(p, m, v, ocore.derive_scalars(hp), 0)
    assert want_idx.size > 100
    spec = layouts.build_spec(W.scaled_dense(layers=1, tp=2))
    pipe = DeltaPipeline(spec, capacity=n)
    pipe.reset()
    pipe.extract(dev(p), dev(m), dev(v), hp)
    sync()
    idx, val, total = pipe.delta()
    assert total == want_idx.size
    assert np.array_equal(idx, want_idx) and np.array_equal(val, want_val)
    pipe.close()


@pytest.mark.parametrize("make", [
    lambda: W.scaled_dense(layers=2, tp=2, lr=1e-6),
    lambda: W.scaled_dense(layers=2, tp=2, lr=1e-4),
    lambda: W.tiny_block(),
])
def test_ordered_extract_is_ascending_and_exact(make):
    """dte_extract_delta_ordered writes exactly the oracle's sorted delta,
    identical bytes on repeated calls, ascending across appended calls."""
    wl = make()
    say("case: ordered extract", wl.name, wl.hp.lr)
    res, st = oracle_state(wl)
    p, m, v = dev(st["p"]), dev(st["m"]), dev(st["v"])
    spec = layouts.build_spec(wl)
    pipe = DeltaPipeline(spec, capacity=max(1, res.idx.size), ordered=True)
    for _ in range(2):
        pipe.reset()
        pipe.extract(p, m, v, wl.hp)
        sync()
        idx, val, total = pipe.delta(raw=True)
        assert total == res.idx.size
        assert np.array_equal(idx, res.idx) and np.array_equal(val, res.val)
    # two appended sub-ranges, the second misaligned and ragged
    cut = (wl.numel // 3) | 1
    pipe.reset()
    pipe.extract(p[:cut], m[:cut], v[:cut], wl.hp, n=cut, index_base=0)
    pipe.extract(p[cut:], m[cut:], v[cut:], wl.hp, n=wl.numel - cut, index_base=cut)
    sync()
    idx, val, total = pipe.delta(raw=True)
    assert total == res.idx.size
    assert np.array_equal(idx, res.idx) and np.array_equal(val, res.val)
    # theta_hat in ordered mode
    prev = torch.empty_like(p)
    pipe.reset()
    pipe.extract(p, m, v, wl.hp, out_prev=prev)
    sync()
    assert np.array_equal(prev.cpu().numpy().view(np.uint32), st["ph"].view(np.uint32))
    idx, val, _ = pipe.delta(raw=True)
    assert np.array_equal(idx, res.idx) and np.array_equal(val, res.val)
    # the ordered delta through remap and apply
    pl = oplan.build_plan(wl)
    pipe.remap()
    sync()
    buckets, counts = pipe.buckets()
    want = oremap.remap(pl, res.idx, res.val)
    for r in range(pl.nranks):
        assert counts[r] == want[r][0].size
        assert np.array_equal(buckets[r][0], want[r][0])
        assert np.array_equal(buckets[r][1], want[r][1])
    pipe.close()


def test_ordered_extract_capacity_overflow_reports_total():
    wl = W.scaled_dense(layers=1, tp=2, lr=1e-4)
    say("case: ordered extract overflow", wl.name)
    res, st = oracle_state(wl)
    p, m, v = dev(st["p"]), dev(st["m"]), dev(st["v"])
    cap = res.idx.size // 3
    pipe = DeltaPipeline(layouts.build_spec(wl), capacity=cap, ordered=True)
    pipe.reset()
    pipe.extract(p, m, v, wl.hp)
    sync()
    assert int(pipe.cursor.item()) == res.idx.size
    pipe.close()


@pytest.mark.parametrize("eps", [1e-8, 1e-13])
def test_literal_order_at_the_proof_guards(eps):
    """Literal order around every bound that decides whether the
    "unchanged" proof may be used (|m| near 2^-100 and 2^64, v near 2^-126
    and 2^100, lrb1 * m near the subnormal range, eps below 2^-40 disabling
    the proof), with weights from tiny to huge: bit-exact delta."""
    say("case: literal guards", eps)
    rng = np.random.default_rng(17)
    mags_m = np.float32([0.0, 2.0 ** -101, 2.0 ** -100, 2.0 ** -99, 2.0 ** -60, 2.0 ** -30,
                         1e-4, 1.0, 2.0 ** 63, 2.0 ** 64, 2.0 ** 65, 3e38])
    mags_v = np.float32([0.0, 2.0 ** -149, 2.0 ** -127, 2.0 ** -126, 2.0 ** -125, 1e-12, 1e-6,
                         1.0, 2.0 ** 99, 2.0 ** 100, 2.0 ** 101, 3e38])
    mags_p = np.float32([0.0, 1e-40, 2.0 ** -100, 1e-30, 1e-10, 0.02, 1.0, 1e20, 2.0 ** 100,
                         1e36, 3e38])
    grid = np.array(np.meshgrid(mags_p, mags_m, mags_v, indexing="ij")).reshape(3, -1)
    k = grid.shape[1]
    reps = 24
    p = np.tile(grid[0], reps).astype(np.float32)
    m = np.tile(grid[1], reps).astype(np.float32)
    v = np.tile(grid[2], reps).astype(np.float32)
    # random signs and a few-ulp jitter so some weights sit near BF16 midpoints
    p *= rng.choice(np.float32([-1, 1]), p.size)
    m *= rng.choice(np.float32([-1, 1]), m.size)
    jit = rng.integers(-3, 4, p.size).astype(np.int64)
    pb = p.view(np.uint32).astype(np.int64)
    mid = (pb & ~0xFFFF) | 0x8000
    pb = np.where(np.arange(p.size) % 2 == 0, mid + jit, pb) & 0xFFFFFFFF
    p = pb.astype(np.uint32).view(np.float32)
    assert p.size == k * reps
    for lr in (1e-7, 1e-4, 0.5):
        hp = W.StepHP(lr=lr, eps=eps, order=W.ORDER_LITERAL)
        want_idx, want_val, _ = ocore.detect(p, m, v, ocore.derive_scalars(hp), 0)
        pipe = DeltaPipeline(layouts.build_spec(W.scaled_dense(layers=1, tp=2)),
                             capacity=p.size)
        pipe.reset()
        pipe.extract(dev(p), dev(m), dev(v), hp)
        sync()
        idx, val, total = pipe.delta()
        assert total == want_idx.size, lr
        assert np.array_equal(idx, want_idx) and np.array_equal(val, want_val), lr
        pipe.close()


@pytest.mark.parametrize("make,order", [
    (lambda: W.scaled_dense(layers=2, tp=2, lr=1e-6), W.ORDER_FOLDED),
    (lambda: W.scaled_dense(layers=2, tp=2, lr=1e-4), W.ORDER_FOLDED),
    (lambda: W.scaled_dense(layers=2, tp=2, lr=1e-4), W.ORDER_LITERAL),
    (lambda: W.tiny_block(), W.ORDER_FOLDED),
    (lambda: W.scaled_moe(synth.word, layers=2, ranks=8, attn_tp=2, experts=16, hidden=64,
                          head_dim=16, expert_intermediate=24, lr=1e-5), W.ORDER_FOLDED),
    (lambda: W.scaled_mcore(trainer_rank=1, receiver_tp=4, vocab=64, lr=1e-5), W.ORDER_FOLDED),
])
def test_fused_extract_remap_equals_oracle(make, order):
    """dte_extract_remap: the buckets (and after apply, the shards) equal the
    oracle's remap of its delta; the changed count equals the delta size."""
    wl = make()
    hp = W.StepHP(lr=wl.hp.lr, order=order)
    say("case: fused extract+remap", wl.name, hp.lr, order)
    if wl.sender.kind == "mcore":
        from oracle import mcore
        twin = W.canonical_twin(wl)
        want_d = mcore.extract(wl, hp)
        pl = oplan.build_plan(twin)
        st_res = orun.extract(twin, hp=hp, keep=("ph", "p"))
    else:
        twin = wl
        want_d = orun.extract(wl, hp=hp)
        pl = oplan.build_plan(wl)
        st_res = orun.extract(wl, hp=hp, keep=("ph", "p"))
    p, m, v = generate_state(wl, hp)
    spec = layouts.build_spec(wl)
    old = oremap.layout(pl, ocore.bf16(orun.flat(st_res.parts, "ph")))
    pipe = DeltaPipeline(spec, capacity=1, rank_capacity=[max(1, n) for n in spec.rank_numel],
                         shards=[dev(x.view(np.int16)) for x in old])
    pipe.step_fused(p, m, v, hp, runs=group_runs(wl, hp))
    sync()
    assert int(pipe.cursor.item()) == want_d.idx.size
    buckets, counts = pipe.buckets()
    want = oremap.remap(pl, want_d.idx, want_d.val)
    expect = oremap.apply([x.copy() for x in old], want)
    for r in range(pl.nranks):
        assert counts[r] == want[r][0].size, r
        assert np.array_equal(buckets[r][0], want[r][0]), r
        assert np.array_equal(buckets[r][1], want[r][1]), r
        assert np.array_equal(host_u16(pipe.shards[r]), expect[r]), r
    pipe.close()


def test_fused_extract_remap_rejects_plans_over_16_ranks():
    wl = W.scaled_dense(layers=1, tp=32, heads_q=32, heads_kv=32, head_dim=8, hidden=64,
                        intermediate=128, vocab=64)
    say("case: fused rejects 32 ranks")
    spec = layouts.build_spec(wl)
    pipe = DeltaPipeline(spec, capacity=16)
    p = torch.zeros(wl.numel, dtype=torch.float32, device="cuda")
    with pytest.raises(B.DteError) as e:
        pipe.extract_remap(p, p, p, wl.hp)
    assert e.value.status == B.DTE_ERR_ARG
    pipe.close()


@pytest.mark.parametrize("slack", [0, 1000])
def test_ordered_extract_when_waves_outgrow_their_regions(slack):
    """All changes in the first half of the range (no moments in the second
    half): with a tight capacity each wave's region holds about the mean
    number of entries per wave, so the waves of the first half write their
    first runs to their regions and the later ones through the shared area;
    the delta must still equal the oracle's, in ascending order.  (50 M
    elements: about 2,300 entries per wave there, regions of about 1,150.)"""
    n = 3 << 24
    hp = W.StepHP(lr=1e-4, weight_decay=0.0)
    sc = ocore.derive_scalars(hp)
    rng = np.random.default_rng(26080455 + 44)
    z = lambda: rng.standard_normal(n, dtype=np.float32)  # noqa: E731
    p_prev = np.float32(0.02) * z()
    m_prev = np.float32(1e-4) * z()
    v_prev = np.abs(np.float32(1e-6) * z())
    g = np.float32(1e-3) * z()
    m_prev[n // 2:] = 0
    g[n // 2:] = 0
    p, m, v = ocore.adamw_forward(p_prev, m_prev, v_prev, g, sc)
    idx, val, _ = ocore.detect(p, m, v, sc)
    say("case: ordered extract, skewed delta", idx.size, slack)
    # (the second half keeps a few changes: draws of -0.0, whose inverse
    # with a zero step is +0.0, a different BF16 pattern)
    assert idx.size > 0 and np.count_nonzero(idx >= n // 2) < 100
    cap = idx.size + slack
    tidx = torch.empty(cap, dtype=torch.int64, device="cuda")
    tval = torch.empty(cap, dtype=torch.int16, device="cuda")
    cur = torch.zeros(1, dtype=torch.int64, device="cuda")
    ws = torch.empty(B.dte_ordered_workspace_bytes(cap), dtype=torch.uint8, device="cuda")
    tp, tm, tv = dev(p), dev(m), dev(v)
    for _ in range(2):
        cur.zero_()
        B.dte_extract_delta_ordered(tp.data_ptr(), tm.data_ptr(), tv.data_ptr(), n, 0, hp,
                                    tidx.data_ptr(), tval.data_ptr(), cap, cur.data_ptr(),
                                    ws.data_ptr(), ws.numel())
        sync()
        assert int(cur.item()) == idx.size
        got_i = tidx[:idx.size].cpu().numpy()
        got_v = tval[:idx.size].cpu().numpy().view(np.uint16)
        assert np.array_equal(got_i, idx) and np.array_equal(got_v, val)
        # white box: the workspace's last 256 bytes hold the shared area's
        # counters (entries, runs); both paths were taken
        shared_entries, shared_runs = ws[-256:-240].cpu().numpy().view(np.int64).tolist()
        assert shared_runs > 0 and 0 < shared_entries < idx.size


@pytest.mark.parametrize("lr", [1e-3, 1e-2])
def test_dense_delta_spanning_many_rounds(lr):
    """A 38M-element model at a learning rate where most elements change:
    every wave scans several tiles and stages far more than its area holds
    between two meetings of its block, so the unordered call mixes
    combined reservations with flushes of single waves; the ordered call
    and the remap follow.  Everything equals the oracle."""
    wl = W.scaled_dense(layers=2, tp=2, hidden=1024, heads_q=8, heads_kv=2, head_dim=128,
                        intermediate=4096, vocab=4096, lr=lr)
    say("case: dense delta", wl.name, wl.numel, lr)
    res = orun.extract(wl)
    assert res.idx.size > wl.numel // 4
    p, m, v = generate_state(wl)
    spec = layouts.build_spec(wl)
    for ordered in (False, True):
        pipe = DeltaPipeline(spec, capacity=wl.numel, ordered=ordered)
        pipe.reset()
        pipe.extract(p, m, v, wl.hp)
        pipe.remap()
        sync()
        if ordered:
            idx, val, total = pipe.delta(raw=True)
            assert total == res.idx.size
            assert np.array_equal(idx, res.idx) and np.array_equal(val, res.val)
        else:
            assert_delta_equal(pipe, res)
        buckets, counts = pipe.buckets()
        want = oremap.remap(oplan.build_plan(wl), res.idx, res.val)
        for r in range(len(want)):
            assert np.array_equal(buckets[r][0], want[r][0]), r
            assert np.array_equal(buckets[r][1], want[r][1]), r
        pipe.close()
    del p, m, v
    torch.cuda.empty_cache()


def straddling_state(sc, n, seed):
    """Weights just below a BF16 rounding midpoint (above one, for negative
    weights) and step terms that carry the reconstruction to within about
    2^-21 relatively of that midpoint, on both sides of it: the elements
    whose change only the exact inverse can settle, mixed with ones an
    approximate bound settles."""
    rng = np.random.default_rng(seed)
    hi = (rng.integers(0x3A00, 0x4000, n, dtype=np.uint32) & 0x7FFF)    # |p| ~ 5e-4 .. 2
    mid = ((hi << 16) | 0x8000).view(np.float32).astype(np.float64)     # midpoint above hi
    gap = np.ldexp(mid, -rng.integers(9, 22, n))                       # 2^-9 .. 2^-21 below it
    p = (mid - gap).astype(np.float32)
    decay = float(sc.decay)
    # theta_hat = (p + u) / decay lands on the midpoint for u = mid decay - p
    target = mid * decay - p.astype(np.float64)
    target *= 1.0 + rng.integers(-48, 49, n) * 2.0 ** -21
    v = (10.0 ** rng.uniform(-12, -4, n)).astype(np.float32)
    den = np.sqrt(v.astype(np.float64) * float(sc.rbc2)) + float(sc.eps)
    m = (target * den / float(sc.lrb1)).astype(np.float32)
    neg = rng.random(n) < 0.5                                          # mirror half of them
    p[neg] = -p[neg]
    m[neg] = -m[neg]
    return p, m, v


@pytest.mark.parametrize("lr", [1e-6, 1e-4, 3e-2])
@pytest.mark.parametrize("order", [W.ORDER_FOLDED, W.ORDER_LITERAL])
def test_step_terms_straddling_the_bf16_midpoint(lr, order):
    """Reconstructions within a few binary32 ulps of a BF16 rounding
    midpoint, on either side: every element parity-checked against the
    oracle, with and without theta_hat requested."""
    say("case: straddling midpoints", lr, order)
    n = (1 << 18) + 77
    hp = W.StepHP(lr=lr, order=order)
    sc = ocore.derive_scalars(hp)
    p, m, v = straddling_state(sc, n, 29)
    want_idx, want_val, want_ph = ocore.detect(p, m, v, sc, 0)
    # the inputs do straddle: both outcomes are common
    assert 0.2 * n < want_idx.size < 0.8 * n, want_idx.size
    spec = layouts.build_spec(W.scaled_dense(layers=1, tp=2))
    pipe = DeltaPipeline(spec, capacity=n)
    for with_prev in (False, True):
        prev = torch.empty(n, dtype=torch.float32, device="cuda") if with_prev else None
        pipe.reset()
        pipe.extract(dev(p), dev(m), dev(v), hp, out_prev=prev)
        sync()
        idx, val, total = pipe.delta()
        assert total == want_idx.size, with_prev
        assert np.array_equal(idx, want_idx) and np.array_equal(val, want_val), with_prev
        if with_prev:
            assert np.array_equal(prev.cpu().numpy().view(np.uint32), want_ph.view(np.uint32))
    pipe.close()


@pytest.mark.parametrize("order", [W.ORDER_FOLDED, W.ORDER_LITERAL])
def test_extract_on_torch_adamw_states(order):
    """The tiny block stepped by torch.optim.AdamW (another trainer's
    rounding of the same step): delta and theta_hat equal the oracle's on
    that state."""
    from oracle import mode_b
    from oracle import run as orun_
    say("case: torch-stepped state", order)
    wl = W.tiny_block()
    hp = W.StepHP(lr=wl.hp.lr, order=order, weight_decay=wl.hp.weight_decay, step=wl.hp.step)
    parts = [mode_b.torch_adamw_step(*orun_.draws(wl, k, 0, t.numel), hp)
             for k, t in enumerate(wl.tensors)]
    p, m, v = (np.concatenate([x[i] for x in parts]) for i in range(3))
    want_idx, want_val, want_ph = ocore.detect(p, m, v, ocore.derive_scalars(hp), 0)
    assert want_idx.size > 1000
    spec = layouts.build_spec(wl)
    pipe = DeltaPipeline(spec, capacity=p.size)
    prev = torch.empty(p.size, dtype=torch.float32, device="cuda")
    pipe.reset()
    pipe.extract(dev(p), dev(m), dev(v), hp, out_prev=prev)
    sync()
    idx, val, total = pipe.delta()
    assert total == want_idx.size
    assert np.array_equal(idx, want_idx) and np.array_equal(val, want_val)
    assert np.array_equal(prev.cpu().numpy().view(np.uint32), want_ph.view(np.uint32))
    pipe.reset()
    pipe.extract(dev(p), dev(m), dev(v), hp)
    sync()
    idx, val, total = pipe.delta()
    assert np.array_equal(idx, want_idx) and np.array_equal(val, want_val)
    pipe.close()


@pytest.mark.parametrize("case", ["small", "below", "exact", "partial"])
def test_unordered_tail_taken_in_chunks(case):
    """The unordered call's last full tiles (1/16 of them, once the waves
    have 16 tiles each) are taken by blocks from a counter in the cursor's
    high bits: just below that size (no tail), at it (whole chunks), above
    it with a partial last chunk, and with a cursor that already holds
    entries (append), the delta equals the oracle's and the cursor ends at
    the exact total."""
    waves = 12 * torch.cuda.get_device_properties(0).multi_processor_count
    tiles = {"small": 15, "below": 16 * waves - 1, "exact": 16 * waves,
             "partial": 16 * waves + 1000}[case]
    say("case: dynamic tail", case, tiles)
    n = tiles * 2048 + 77
    rng = np.random.default_rng(tiles)
    p = (rng.standard_normal(n) * 0.02).astype(np.float32)
    m = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    v = np.abs(rng.standard_normal(n) * 1e-6).astype(np.float32)
    hp = W.StepHP(lr=1e-4)
    want_idx, want_val, _ = ocore.detect(p, m, v, ocore.derive_scalars(hp), 100)
    assert want_idx.size > 0
    cap = want_idx.size + 16
    idx = torch.full((cap,), -1, dtype=torch.int64, device="cuda")
    val = torch.zeros(cap, dtype=torch.int16, device="cuda")
    cursor = torch.tensor([5], dtype=torch.int64, device="cuda")
    dp, dm, dv = dev(p), dev(m), dev(v)
    B.dte_extract_delta(dp.data_ptr(), dm.data_ptr(), dv.data_ptr(), n, 100, hp,
                        idx.data_ptr(), val.data_ptr(), cap, cursor.data_ptr(), 0,
                        torch.cuda.current_stream().cuda_stream)
    sync()
    assert int(cursor.item()) == 5 + want_idx.size
    got_i = idx.cpu().numpy()
    assert (got_i[:5] == -1).all()                         # entries before the cursor kept
    got_v = val.cpu().numpy().view(np.uint16)[5:5 + want_idx.size]
    got_i = got_i[5:5 + want_idx.size]
    order = np.argsort(got_i)
    assert np.array_equal(got_i[order], want_idx) and np.array_equal(got_v[order], want_val)
    if case == "partial":
        # a second call appending to the same cursor (the next range of a
        # shard with the same data) starts from a cleared cursor
        idx2 = torch.full((2 * cap,), -1, dtype=torch.int64, device="cuda")
        val2 = torch.zeros(2 * cap, dtype=torch.int16, device="cuda")
        cursor.fill_(0)
        for base in (100, 100 + n):
            B.dte_extract_delta(dp.data_ptr(), dm.data_ptr(), dv.data_ptr(), n, base, hp,
                                idx2.data_ptr(), val2.data_ptr(), 2 * cap, cursor.data_ptr(), 0,
                                torch.cuda.current_stream().cuda_stream)
        sync()
        k = want_idx.size
        assert int(cursor.item()) == 2 * k
        got_i = idx2.cpu().numpy()[:2 * k]
        got_v = val2.cpu().numpy().view(np.uint16)[:2 * k]
        order = np.argsort(got_i)
        assert np.array_equal(got_i[order], np.concatenate([want_idx, want_idx + n]))
        assert np.array_equal(got_v[order], np.concatenate([want_val, want_val]))
