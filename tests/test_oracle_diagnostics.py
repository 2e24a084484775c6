"""Pins of the oracle's reconstruction diagnostics.

The inverse of sec. 4.1 (eq. adamw_inverse) is a numerical reconstruction
of the previous weights, not a bitwise recovery, so beside the delta the
oracle reports four per-element counts against the true pre-step weights
theta_{t-1}: binary32 patterns that differ, BF16 patterns that differ
(b(theta_hat) != b(theta_{t-1})), true BF16 changes (b(theta_{t-1}) !=
b(theta_t)), and elements a receiver holding b(theta_{t-1}) keeps stale.

The expected counts come from an evaluator written here that shares
nothing with the oracle:
  * the step scalars are exact rationals rounded once to binary32;
  * every binary32 operation is evaluated in binary64 and rounded once,
    which is exact for + - * / and sqrt of binary32 operands (53 >= 2*24 + 2,
    the double-rounding theorem);
  * BF16 quantisation rounds the exact value to 8 significant bits, ties to
    even (Python's round of a Fraction), and compares (sign, value).
A hand-built state puts pre-step weights on BF16 rounding midpoints (and
one binary32 ulp either side of them) at the top of a binade, with a step
term that carries the forward step across the binade boundary; there the
forward step's rounding error is a whole ulp of the pre-step weight, so the
reconstruction lands on the other side of the midpoint for a set of
elements known before the oracle runs.  The oracle's windowed,
multi-threaded driver must report exactly the evaluator's counts; planted
mistakes in the oracle (a comparison against b(theta_t), a dropped window)
must change them.
"""
import math
import random
import struct
from fractions import Fraction

import numpy as np
import pytest

import synth
from oracle import run as orun
from synth import workloads as W


def f32(x):
    return struct.unpack("<f", struct.pack("<f", x))[0]


def f32_bits(x):
    return struct.unpack("<I", struct.pack("<f", x))[0]


def from_bits(b):
    return struct.unpack("<f", struct.pack("<I", b))[0]


class Evaluator:
    """Folded-order AdamW step and inverse (sec. 4.1; appendix A), one
    binary32 rounding per operation."""

    def __init__(self, hp):
        lr, wd = Fraction(hp.lr), Fraction(hp.weight_decay)
        b1, b2 = Fraction(hp.beta1), Fraction(hp.beta2)
        self.lrb1 = f32(float(lr / (1 - b1 ** hp.step)))
        self.rbc2 = f32(float(1 / (1 - b2 ** hp.step)))
        self.eps = f32(float(Fraction(hp.eps)))
        self.decay = f32(float(1 - lr * wd))
        self.b1, self.b2 = f32(float(b1)), f32(float(b2))
        self.omb1, self.omb2 = f32(float(1 - b1)), f32(float(1 - b2))

    def step_term(self, m, v):
        s = f32(math.sqrt(f32(v * self.rbc2)))
        return f32(f32(self.lrb1 * m) / f32(s + self.eps))

    def forward(self, p_prev, m_prev, v_prev, g):
        m = f32(f32(self.b1 * m_prev) + f32(self.omb1 * g))
        v = f32(f32(self.b2 * v_prev) + f32(self.omb2 * f32(g * g)))
        return f32(f32(self.decay * p_prev) - self.step_term(m, v)), m, v

    def post_step(self, p_prev, m, v):
        """theta_t from theta_{t-1} and the post-step moments."""
        return f32(f32(self.decay * p_prev) - self.step_term(m, v))

    def inverse(self, p, m, v):
        return f32(f32(p + self.step_term(m, v)) / self.decay)


def bf16(x):
    """(sign, value) of x rounded to BF16: 8 significant bits, ties to even,
    exponent range of binary32 (subnormals on the same grid), overflow to
    infinity."""
    sign = math.copysign(1.0, x)
    if x == 0:
        return sign, Fraction(0)
    _, e2 = math.frexp(abs(x))
    e = max(e2 - 1, -126)
    quantum = Fraction(2) ** (e - 7)
    val = round(Fraction(abs(x)) / quantum) * quantum
    if val >= Fraction(2) ** 128:
        return sign, math.inf
    return sign, val


def expected_counts(p_prev, p, m, v, ev):
    """The five counts, element by element, with the evaluator above."""
    c = dict(n=0, changed=0, fp32_recon_mismatch=0, bf16_recon_mismatch=0, true_changed=0,
             apply_vs_prev_diff=0)
    for a, b, mm, vv in zip(p_prev.tolist(), p.tolist(), m.tolist(), v.tolist()):
        ph = ev.inverse(b, mm, vv)
        q_prev, q_ph, q_p = bf16(a), bf16(ph), bf16(b)
        c["n"] += 1
        c["changed"] += q_ph != q_p
        c["fp32_recon_mismatch"] += f32_bits(ph) != f32_bits(a)
        c["bf16_recon_mismatch"] += q_ph != q_prev
        c["true_changed"] += q_prev != q_p
        c["apply_vs_prev_diff"] += (q_prev != q_ph) and (q_ph == q_p)
    return c


def as_dict(d):
    return {k: getattr(d, k) for k in ("n", "changed", "fp32_recon_mismatch",
                                       "bf16_recon_mismatch", "true_changed",
                                       "apply_vs_prev_diff")}


HP = W.StepHP(lr=1e-4)          # DECAY != 1: every rounding of the inverse is live


def planted_element(rng, ev):
    """A pre-step weight on (or one ulp beside) a BF16 midpoint with the
    largest 7-bit BF16 significand, and post-step moments whose step term
    pushes theta_t = DECAY theta_{t-1} - u into the next binade."""
    e = rng.randrange(-9, -4)
    sign = rng.randrange(2)
    hi = (sign << 15) | ((e + 127) << 7) | 0x7F
    p_prev = from_bits((hi << 16) | rng.choice((0x8000, 0x7FFF, 0x8001)))
    v = f32(rng.uniform(0.5e-6, 2e-6))
    target = 2.0 ** (e - 8) * rng.uniform(0.8, 4.0)      # |u| above half a BF16 ulp
    m = f32(-math.copysign(1.0, p_prev) * target / ev.lrb1 * math.sqrt(v * ev.rbc2))
    return p_prev, ev.post_step(p_prev, m, v), m, v


def build_fixture(sizes, planted_per_tensor, seed=7):
    """Per tensor (p_prev, p, m, v) as binary32 arrays, and the positions of
    the planted elements whose BF16 reconstruction differs (found with the
    evaluator before the oracle runs)."""
    ev = Evaluator(HP)
    rng = random.Random(seed)
    nrng = np.random.default_rng(seed)
    tensors, planted = [], []
    for k, n in enumerate(sizes):
        p_prev = (nrng.standard_normal(n) * 0.02).astype(np.float32)
        m_prev = (nrng.standard_normal(n) * 1e-4).astype(np.float32)
        v_prev = np.abs(nrng.standard_normal(n) * 1e-6).astype(np.float32)
        g = (nrng.standard_normal(n) * 1e-3).astype(np.float32)
        p, m, v = (np.empty(n, np.float32) for _ in range(3))
        for i in range(n):
            if i % 5 == 4:                   # untouched: zero moments and gradient
                m_prev[i] = v_prev[i] = g[i] = 0.0
            p[i], m[i], v[i] = ev.forward(float(p_prev[i]), float(m_prev[i]), float(v_prev[i]),
                                          float(g[i]))
        spots = sorted(rng.sample(range(n), planted_per_tensor))
        hits = []
        for i in spots:
            while True:
                a, b, mm, vv = planted_element(rng, ev)
                if bf16(ev.inverse(b, mm, vv)) != bf16(a):
                    break
            p_prev[i], p[i], m[i], v[i] = a, b, mm, vv
            hits.append(i)
        tensors.append((p_prev, p, m, v))
        planted.append(hits)
    return tensors, planted, ev


SIZES = (3001, 4096, 1537, 2777)


@pytest.fixture(scope="module")
def fixture():
    tensors, planted, ev = build_fixture(SIZES, planted_per_tensor=9)
    wl = W.Workload("diag_fixture", "hand-built state", 1, W.ModelDims(8, 1, 1, 8),
                    tuple(W.Tensor("t%d" % k, (n,), "q") for k, n in enumerate(SIZES)), HP,
                    W.Receiver("tp", tp=1))
    want = dict(n=0, changed=0, fp32_recon_mismatch=0, bf16_recon_mismatch=0, true_changed=0,
                apply_vs_prev_diff=0)
    for arrs in tensors:
        for key, x in expected_counts(*arrs, ev).items():
            want[key] += x
    return wl, tensors, planted, want


def serve(tensors):
    def state(wl, k, lo, hi, sc, threads=1):
        return tuple(a[lo:hi].copy() for a in tensors[k])
    return state


def test_fixture_is_what_it_claims(fixture):
    """Every planted element sits at a BF16 midpoint or one ulp beside it,
    and its reconstruction lies on the other side; the counts are not
    degenerate."""
    wl, tensors, planted, want = fixture
    ev = Evaluator(HP)
    for (p_prev, p, m, v), hits in zip(tensors, planted):
        for i in hits:
            low = f32_bits(float(p_prev[i])) & 0xFFFF
            assert low in (0x7FFF, 0x8000, 0x8001)
            assert bf16(ev.inverse(float(p[i]), float(m[i]), float(v[i]))) != \
                bf16(float(p_prev[i]))
    n_planted = sum(len(h) for h in planted)
    assert n_planted == 36
    assert want["bf16_recon_mismatch"] >= n_planted
    assert want["fp32_recon_mismatch"] >= want["bf16_recon_mismatch"]
    assert want["changed"] > 100 and want["true_changed"] > 100
    assert want["apply_vs_prev_diff"] > 0


@pytest.mark.parametrize("threads,window", [(1, 1 << 20), (4, 700), (3, 257)])
def test_oracle_counts_equal_elementwise_counts(fixture, monkeypatch, threads, window):
    wl, tensors, planted, want = fixture
    monkeypatch.setattr(orun, "state", serve(tensors))
    got = orun.extract(wl, threads=threads, max_window=window)
    assert as_dict(got.diag) == want


def test_planted_comparison_against_theta_t_is_caught(fixture, monkeypatch):
    """An oracle that compared b(theta_hat) with b(theta_t) instead of
    b(theta_{t-1}) would not pass the check above."""
    wl, tensors, planted, want = fixture
    monkeypatch.setattr(orun, "state", serve(tensors))
    real = orun.count_diagnostics

    def wrong(p_prev, ph, p, changed):
        return real(p, ph, p, changed)

    monkeypatch.setattr(orun, "count_diagnostics", wrong)
    got = as_dict(orun.extract(wl, threads=4, max_window=700).diag)
    assert got["bf16_recon_mismatch"] != want["bf16_recon_mismatch"]


def test_planted_dropped_window_is_caught(fixture, monkeypatch):
    """An oracle that skipped one window (here the one holding the first
    planted element of the second tensor) would not pass the check above."""
    wl, tensors, planted, want = fixture
    monkeypatch.setattr(orun, "state", serve(tensors))
    real = orun.windows
    victim = planted[1][0]

    def drop(wl_, max_window=1 << 24, tensors=None):
        return [w for w in real(wl_, max_window, tensors)
                if not (w.tensor == 1 and w.lo <= victim < w.hi)]

    monkeypatch.setattr(orun, "windows", drop)
    got = as_dict(orun.extract(wl, threads=4, max_window=700).diag)
    assert got["bf16_recon_mismatch"] < want["bf16_recon_mismatch"]
    assert got["n"] < want["n"]


def test_counts_on_generated_state():
    """The oracle's counts on windows of a generated dense model (the
    shared input generator's draws, every tensor kind) equal the
    evaluator's element-by-element counts."""
    wl = W.scaled_dense(layers=1, tp=2, lr=1e-4)
    ev = Evaluator(wl.hp)
    rng = np.random.default_rng(3)
    wins = []
    for k, t in enumerate(wl.tensors):
        n = min(t.numel, 2500)
        lo = int(rng.integers(0, t.numel - n + 1))
        wins.append(orun.Window(k, lo, lo + n))
    want = dict(n=0, changed=0, fp32_recon_mismatch=0, bf16_recon_mismatch=0, true_changed=0,
                apply_vs_prev_diff=0)
    for w in wins:
        n = w.hi - w.lo
        draws = [synth.draw_cpu(n, wl.seed, w.tensor, kind, w.lo)
                 for kind in (W.KIND_P_PREV, W.KIND_M_PREV, W.KIND_V_PREV, W.KIND_GRAD)]
        p_prev = draws[0]
        p, m, v = (np.empty(n, np.float32) for _ in range(3))
        for i in range(n):
            p[i], m[i], v[i] = ev.forward(*(float(d[i]) for d in draws))
        for key, x in expected_counts(p_prev, p, m, v, ev).items():
            want[key] += x
    got = orun.extract(wl, wins=wins, threads=4)
    assert as_dict(got.diag) == want
    assert want["fp32_recon_mismatch"] > 0 and want["changed"] > 0
