"""Pins of the oracle's binary32 arithmetic (sec. 4.1, appendix A).

Against: exact rational evaluation of the step scalars and of the paper's
inverse (eq. adamw_inverse), torch.optim.AdamW for the forward step, the
round-trip invariant inverse(forward(x)) ~ x (exact in exact arithmetic,
sec. 4.1), and closed-form special cases.  A per-operation binary64
evaluation rounded to binary32 (exact for + - * / sqrt by the double-
rounding theorem, 53 >= 2*24 + 2) checks the C build itself: no fused
multiply-add, no flushed subnormals, correctly rounded divide and sqrt.
"""
import math
import struct
from decimal import Decimal, getcontext
from fractions import Fraction

import numpy as np
import pytest
import torch

import synth
from oracle import core
from synth import workloads as W

HP = W.StepHP(lr=1e-6)


def f32(x):
    return struct.unpack("<f", struct.pack("<f", x))[0]


def f32_bits(x):
    return struct.unpack("<I", struct.pack("<f", x))[0]


def _exact_scalars(hp):
    b1, b2 = Fraction(hp.beta1), Fraction(hp.beta2)
    lr, wd = Fraction(hp.lr), Fraction(hp.weight_decay)
    return {"lrb1": lr / (1 - b1 ** hp.step), "rbc2": 1 / (1 - b2 ** hp.step),
            "eps": Fraction(hp.eps), "decay": 1 - lr * wd}


@pytest.mark.parametrize("lr", [0.0, 1e-7, 1e-6, 1e-5, 1e-4, 1e-3])
@pytest.mark.parametrize("step", [1, 2, 100, 10000])
def test_scalars_are_exact_values_rounded_once(lr, step):
    hp = W.StepHP(lr=lr, step=step)
    sc = core.derive_scalars(hp)
    ex = _exact_scalars(hp)
    for name in ("lrb1", "rbc2", "eps", "decay"):
        want = f32(float(ex[name]))
        assert f32_bits(getattr(sc, name)) == f32_bits(want), (name, lr, step)


def test_scalar_values_at_step_100():
    sc = core.derive_scalars(HP)
    assert abs(sc.lrb1 - 1.0000266e-6) < 1e-12
    assert abs(sc.rbc2 - 10.503335) < 1e-5
    assert sc.decay == 1.0            # 1 - 1e-8 rounds to 1.0f
    sc4 = core.derive_scalars(W.StepHP(lr=1e-4))
    assert f32_bits(sc4.decay) == f32_bits(1.0 - 17 * 2.0 ** -24)


def _state(n, seed=5, scale_m=1.0):
    p_prev = synth.draw_cpu(n, seed, 0, W.KIND_P_PREV)
    m_prev = synth.draw_cpu(n, seed, 0, W.KIND_M_PREV) * np.float32(scale_m)
    v_prev = synth.draw_cpu(n, seed, 0, W.KIND_V_PREV)
    g = synth.draw_cpu(n, seed, 0, W.KIND_GRAD)
    return p_prev, m_prev, v_prev, g


@pytest.mark.parametrize("lr", [1e-6, 1e-4, 1e-2])
def test_forward_matches_torch_adamw(lr):
    """One AdamW step of the oracle vs torch.optim.AdamW from step t-1."""
    hp = W.StepHP(lr=lr)
    n = 4096
    p_prev, m_prev, v_prev, g = _state(n)
    sc = core.derive_scalars(hp)
    p, m, v = core.adamw_forward(p_prev, m_prev, v_prev, g, sc)

    param = torch.nn.Parameter(torch.from_numpy(p_prev.copy()))
    opt = torch.optim.AdamW([param], lr=lr, betas=(hp.beta1, hp.beta2), eps=hp.eps,
                            weight_decay=hp.weight_decay, foreach=False, fused=False)
    param.grad = torch.from_numpy(g.copy())
    opt.state[param] = {"step": torch.tensor(float(hp.step - 1)),
                        "exp_avg": torch.from_numpy(m_prev.copy()),
                        "exp_avg_sq": torch.from_numpy(v_prev.copy())}
    opt.step()
    tp = param.detach().numpy()
    tm = opt.state[param]["exp_avg"].numpy()
    tv = opt.state[param]["exp_avg_sq"].numpy()
    # The two evaluation orders differ by a few roundings of the *terms*
    # (m and p are sums whose terms can cancel), so the tolerance is a few
    # ulp of the largest term, not of the result.
    ulp = lambda *xs: np.spacing(np.max(np.abs(np.stack(xs)), axis=0).astype(np.float32))  # noqa
    b1, b2 = np.float32(hp.beta1), np.float32(hp.beta2)
    u = np.float32(sc.decay) * p_prev - p
    assert np.all(np.abs(m - tm) <= 2 * ulp(b1 * m_prev, g * np.float32(0.1)))
    assert np.all(np.abs(v - tv) <= 2 * ulp(b2 * v_prev, g * g * np.float32(1e-3)))
    assert np.all(np.abs(p - tp) <= 4 * ulp(p_prev, u))
    # the update moved the weights (a sign error would still be caught here)
    assert np.count_nonzero(p != p_prev) > n // 2


def _dsqrt(x: Fraction) -> Fraction:
    getcontext().prec = 80
    d = Decimal(x.numerator) / Decimal(x.denominator)
    return Fraction(d.sqrt())


def _exact_inverse(p, m, v, ex):
    """The paper's eq. adamw_inverse in exact arithmetic on binary32 inputs."""
    m_hat = Fraction(m) * (1 / (ex["lrb1_den"]))
    v_hat = Fraction(v) * ex["rbc2"]
    upd = ex["lr"] * m_hat / (_dsqrt(v_hat) + ex["eps"])
    return (Fraction(p) + upd) / ex["decay"]


@pytest.mark.parametrize("lr", [1e-6, 1e-4, 1e-2])
def test_inverse_within_bound_of_exact(lr):
    """ph agrees with the exact inverse of the binary32 state within the
    error budget of the folded order: u carries a relative error of at most
    about 6 * 2^-24 (rounded LRB1, the product, v*RBC2, sqrt, + EPS, the
    quotient); n = p + u and ph = n / DECAY add a half-ulp each, and the
    rounded DECAY at most one ulp of ph."""
    hp = W.StepHP(lr=lr)
    sc = core.derive_scalars(hp)
    n = 3000
    p_prev, m_prev, v_prev, g = _state(n, seed=11)
    p, m, v = core.adamw_forward(p_prev, m_prev, v_prev, g, sc)
    ph = core.invert(p, m, v, sc)
    ex = _exact_scalars(hp)
    ex["lr"] = Fraction(hp.lr)
    ex["lrb1_den"] = 1 - Fraction(hp.beta1) ** hp.step
    for i in range(n):
        want = _exact_inverse(float(p[i]), float(m[i]), float(v[i]), ex)
        err = abs(Fraction(float(ph[i])) - want)
        ulp = Fraction(float(np.spacing(np.float32(abs(float(want))))))
        u = abs(want * ex["decay"] - Fraction(float(p[i])))
        bound = 2 * ulp + 8 * u * Fraction(1, 1 << 24) / ex["decay"]
        assert err <= bound, (i, float(ph[i]), float(want))


@pytest.mark.parametrize("lr", [1e-7, 1e-6, 1e-5, 1e-4])
def test_round_trip_recovers_previous_weights(lr):
    """Inverse after forward returns p_prev up to rounding (sec. 4.1: exact
    in exact arithmetic): within 2 ulp of the larger of |p_prev| and the
    step |p - p_prev|, and mostly bit-exact."""
    hp = W.StepHP(lr=lr)
    sc = core.derive_scalars(hp)
    n = 1 << 18
    p_prev, m_prev, v_prev, g = _state(n, seed=21)
    p, m, v = core.adamw_forward(p_prev, m_prev, v_prev, g, sc)
    ph = core.invert(p, m, v, sc)
    scale = np.maximum(np.abs(p_prev), np.abs(p - p_prev))
    assert np.all(np.abs(ph - p_prev) <= 2 * np.spacing(scale))
    assert np.count_nonzero(ph != p_prev) < n * 0.01


def test_special_cases():
    n = 1 << 14
    p_prev, m_prev, v_prev, g = _state(n, seed=31)
    # lr = 0: the step changes nothing and the inverse is the identity
    sc0 = core.derive_scalars(W.StepHP(lr=0.0))
    p, m, v = core.adamw_forward(p_prev, m_prev, v_prev, g, sc0)
    assert np.array_equal(p.view(np.uint32), p_prev.view(np.uint32))
    assert np.array_equal(core.invert(p, m, v, sc0).view(np.uint32), p.view(np.uint32))
    # zero moments: u = 0, so ph = p / DECAY with one rounding
    sc = core.derive_scalars(W.StepHP(lr=1e-4))
    z = np.zeros(n, np.float32)
    ph = core.invert(p_prev, z, z, sc)
    assert np.array_equal(ph.view(np.uint32), (p_prev / np.float32(sc.decay)).view(np.uint32))
    # no weight decay: DECAY = 1 and ph = fl(p + u)
    scw = core.derive_scalars(W.StepHP(lr=1e-4, weight_decay=0.0))
    assert scw.decay == 1.0
    # untouched element (m = v = g = 0): forward is p = DECAY * p_prev
    p, m, v = core.adamw_forward(p_prev, z, z, z, sc)
    assert np.array_equal(p.view(np.uint32), (np.float32(sc.decay) * p_prev).view(np.uint32))
    assert not m.any() and not v.any()


def _bruteforce_inverse(p, m, v, s):
    out = []
    for pi, mi, vi in zip(p.tolist(), m.tolist(), v.tolist()):
        vh = f32(vi * s.rbc2)
        sq = f32(math.sqrt(vh))
        den = f32(sq + s.eps)
        num = f32(s.lrb1 * mi)
        u = f32(num / den)
        out.append(f32(f32(pi + u) / s.decay))
    return np.array(out, np.float32)


def test_c_build_rounds_every_operation():
    """The C build evaluates each operation with one IEEE rounding (no FMA
    contraction, subnormals kept): compare with binary64-then-round."""
    rng = np.random.default_rng(7)
    n = 20000
    sc = core.derive_scalars(W.StepHP(lr=1e-4))
    p = (rng.standard_normal(n) * 0.02).astype(np.float32)
    m = (rng.standard_normal(n) * 1e-4).astype(np.float32)
    v = np.abs(rng.standard_normal(n) * 1e-6).astype(np.float32)
    # subnormal and extreme magnitudes
    p[:8] = np.array([1e-45, -1e-45, 1e-39, -3e-39, 0.0, -0.0, 3e38, -3e38], np.float32)
    m[8:16] = np.array([1e-45, -1e-40, 0.0, 1e-20, -1e-30, 2e-38, 1.0, -1.0], np.float32)
    v[16:24] = np.array([0.0, 1e-45, 1e-40, 1e-38, 1e-30, 1.0, 100.0, 1e-20], np.float32)
    got = core.invert(p, m, v, sc)
    want = _bruteforce_inverse(p, m, v, sc)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


# -- literal operation order (eq. adamw_inverse as printed) -----------------

LIT = W.ORDER_LITERAL


@pytest.mark.parametrize("lr", [0.0, 1e-6, 1e-4])
@pytest.mark.parametrize("step", [1, 100, 10000])
def test_literal_scalars_are_exact_values_rounded_once(lr, step):
    hp = W.StepHP(lr=lr, step=step, order=LIT)
    sc = core.derive_scalars(hp)
    assert sc.order == 1
    b1, b2 = Fraction(hp.beta1), Fraction(hp.beta2)
    want = {"lr": Fraction(lr), "bc1": 1 - b1 ** step, "bc2": 1 - b2 ** step}
    for name, x in want.items():
        assert f32_bits(getattr(sc, name)) == f32_bits(f32(float(x))), name


def _bruteforce_literal(p, m, v, s):
    out = []
    for pi, mi, vi in zip(p.tolist(), m.tolist(), v.tolist()):
        mh = f32(mi / s.bc1)
        vq = f32(vi / s.bc2)
        d = f32(f32(math.sqrt(vq)) + s.eps)
        u = f32(s.lr * f32(mh / d))
        out.append(f32(f32(pi + u) / s.decay))
    return np.array(out, np.float32)


def test_c_build_literal_rounds_every_operation():
    rng = np.random.default_rng(8)
    n = 20000
    sc = core.derive_scalars(W.StepHP(lr=1e-4, order=LIT))
    p = (rng.standard_normal(n) * 0.02).astype(np.float32)
    m = (rng.standard_normal(n) * 1e-4).astype(np.float32)
    v = np.abs(rng.standard_normal(n) * 1e-6).astype(np.float32)
    p[:8] = np.array([1e-45, -1e-45, 1e-39, -3e-39, 0.0, -0.0, 3e38, -3e38], np.float32)
    m[8:16] = np.array([1e-45, -1e-40, 0.0, 1e-20, -1e-30, 2e-38, 1.0, -1.0], np.float32)
    v[16:24] = np.array([0.0, 1e-45, 1e-40, 1e-38, 1e-30, 1.0, 100.0, 1e-20], np.float32)
    got = core.invert(p, m, v, sc)
    want = _bruteforce_literal(p, m, v, sc)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


@pytest.mark.parametrize("lr", [1e-6, 1e-4, 1e-2])
def test_literal_inverse_within_bound_of_exact(lr):
    """The literal order against exact eq. adamw_inverse: u carries at most
    about 9 roundings (LR, BC1, m/BC1, BC2, v/BC2, sqrt, + EPS, the ratio,
    the product); then the same half-ulps as the folded order."""
    hp = W.StepHP(lr=lr, order=LIT)
    sc = core.derive_scalars(hp)
    n = 3000
    p_prev, m_prev, v_prev, g = _state(n, seed=12)
    p, m, v = core.adamw_forward(p_prev, m_prev, v_prev, g, sc)
    ph = core.invert(p, m, v, sc)
    ex = _exact_scalars(hp)
    ex["lr"] = Fraction(hp.lr)
    ex["lrb1_den"] = 1 - Fraction(hp.beta1) ** hp.step
    for i in range(n):
        want = _exact_inverse(float(p[i]), float(m[i]), float(v[i]), ex)
        err = abs(Fraction(float(ph[i])) - want)
        ulp = Fraction(float(np.spacing(np.float32(abs(float(want))))))
        u = abs(want * ex["decay"] - Fraction(float(p[i])))
        bound = 2 * ulp + 10 * u * Fraction(1, 1 << 24) / ex["decay"]
        assert err <= bound, (i, float(ph[i]), float(want))


@pytest.mark.parametrize("lr", [1e-6, 1e-4])
def test_literal_round_trip_and_difference_from_folded(lr):
    n = 1 << 16
    p_prev, m_prev, v_prev, g = _state(n, seed=22)
    lit = core.derive_scalars(W.StepHP(lr=lr, order=LIT))
    fol = core.derive_scalars(W.StepHP(lr=lr))
    p, m, v = core.adamw_forward(p_prev, m_prev, v_prev, g, lit)
    ph = core.invert(p, m, v, lit)
    scale = np.maximum(np.abs(p_prev), np.abs(p - p_prev))
    assert np.all(np.abs(ph - p_prev) <= 2 * np.spacing(scale))
    # the two orders round differently somewhere, and stay within 2 ulp
    pf, _, _ = core.adamw_forward(p_prev, m_prev, v_prev, g, fol)
    assert np.count_nonzero(pf != p) > 0
    assert np.all(np.abs(pf - p) <= 2 * np.spacing(np.maximum(np.abs(p), np.abs(p - p_prev))))
