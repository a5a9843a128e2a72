"""Pins of the oracle's LAMB step and its exact fp32 sum of squares.

LAMB (You et al.) is listed in ZeRO's related work (Sec. 2.3, training
optimizers) among the adaptive optimizers whose memory ZeRO's partitioning
reduces.  Nothing here retypes the oracle's formulas.  The exact sum of squares
is checked against Python's exact integer and rational arithmetic and against
math.fsum (a correctly rounded sum of the exactly representable float64
squares).  The step is checked against the properties that define LAMB: its
moments are Adam's; each layer's update has norm lr * phi(||theta||); the
update is invariant to a power-of-two rescaling of a layer; a zero layer takes
Adam's step; a zero gradient with weight decay shrinks the layer by (1 - lr);
layers are independent.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle

HP = dict(beta1=0.9, beta2=0.999, eps=1e-8)


def exact_sumsq(x: np.ndarray) -> float:
    """Sum of squares with Python's exact rationals, rounded once by float()."""
    total = Fraction(0)
    for a in x.astype(np.float64).tolist():
        f = Fraction(a)
        total += f * f
    return float(total)


def random_finite_f32(rng, n):
    bits = rng.integers(0, 1 << 32, size=n, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    return np.where(np.isfinite(x), x, np.float32(1.5)).astype(np.float32)


# --------------------------------------------------------------------------
# exact sum of squares
# --------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(6))
def test_sumsq_equals_exact_rational_sum(seed):
    rng = np.random.default_rng(seed)
    for n in (1, 2, 7, 64, 1000):
        x = random_finite_f32(rng, n)  # every exponent, subnormals included
        assert oracle.sumsq_f32(x) == exact_sumsq(x)


def test_sumsq_equals_fsum_of_float64_squares():
    # A float32 square is exact in float64, and math.fsum returns the correctly
    # rounded sum of its float64 inputs.
    rng = np.random.default_rng(11)
    for scale in (1e-30, 1e-3, 1.0, 1e10, 1e18):
        x = (rng.standard_normal(200_000) * scale).astype(np.float32)
        sq = x.astype(np.float64) ** 2
        assert oracle.sumsq_f32(x) == math.fsum(sq.tolist())
    x = np.concatenate([rng.standard_normal(1000) * 1e15, rng.standard_normal(100_000) * 1e-3]).astype(np.float32)
    rng.shuffle(x)
    assert oracle.sumsq_f32(x) == math.fsum((x.astype(np.float64) ** 2).tolist())


def test_sumsq_rounding_ties_and_sticky_bits():
    # 2^60 + 128 is halfway between two doubles (spacing 256): ties go to even
    assert oracle.sumsq_f32(np.array([2.0 ** 30, 8, 8], np.float32)) == 2.0 ** 60
    # 2^60 + 256 + 128: halfway again, the even neighbour is above
    assert oracle.sumsq_f32(np.array([2.0 ** 30, 16, 8, 8], np.float32)) == 2.0 ** 60 + 512
    # 2^60 + 128 + 2^-10: just above halfway, decided by a bit far below the kept ones
    assert oracle.sumsq_f32(np.array([2.0 ** 30, 8, 8, 2.0 ** -5], np.float32)) == 2.0 ** 60 + 256
    # a naive float64 running sum of the same squares loses the small terms entirely
    naive = 0.0
    for a in (2.0 ** 30, 8.0, 8.0, 1.0):
        naive += a * a
    assert naive == 2.0 ** 60 and oracle.sumsq_f32(np.array([2.0 ** 30, 8, 8, 1], np.float32)) == 2.0 ** 60 + 256


@pytest.mark.parametrize("q", range(0, 7))
def test_sumsq_carries_across_words(q):
    # squares whose bits end exactly at the top of a 64-bit word: two of them carry
    # into the next word; many of them carry further
    e = (64 * q + 80 - 298) // 2
    x = np.float32(math.ldexp((1 << 24) - 1, e))
    assert np.isfinite(x) and x != 0
    for k in (2, 3, 1000):
        arr = np.full(k, x, np.float32)
        assert oracle.sumsq_f32(arr) == exact_sumsq(arr)


@pytest.mark.parametrize("q", range(0, 6))
def test_sumsq_carry_through_a_full_word(q):
    # Fill word q+1 of the accumulator (unit 2^-298) with ones from squares of powers of
    # two (2^j is a square for even j and the sum of two equal squares for odd j), then
    # let four squares overflow word q: the carry must run through the full word.
    vals = []
    for j in range(64):
        b = 64 * (q + 1) + j - 298
        if j % 2 == 0:
            vals.append(math.ldexp(1.0, b // 2))
        else:
            vals += [math.ldexp(1.0, (b - 1) // 2)] * 2
    vals += [math.ldexp(1.0, (64 * q + 62 - 298) // 2)] * 4
    arr = np.array(vals, np.float32)
    assert np.all(np.isfinite(arr)) and np.all(arr.astype(np.float64) == np.array(vals))
    assert oracle.sumsq_f32(arr) == exact_sumsq(arr)


def test_sumsq_special_values():
    assert oracle.sumsq_f32(np.zeros(0, np.float32)) == 0.0
    assert oracle.sumsq_f32(np.array([0.0, -0.0], np.float32)) == 0.0
    tiny = np.float32(np.finfo(np.float32).smallest_subnormal)
    assert oracle.sumsq_f32(np.array([tiny], np.float32)) == 2.0 ** -298
    big = np.float32(np.finfo(np.float32).max)
    assert oracle.sumsq_f32(np.array([big] * 3, np.float32)) == exact_sumsq(np.array([big] * 3, np.float32))
    assert oracle.sumsq_f32(np.array([1.0, np.inf], np.float32)) == math.inf
    assert oracle.sumsq_f32(np.array([1.0, -np.inf], np.float32)) == math.inf
    assert math.isnan(oracle.sumsq_f32(np.array([np.inf, np.nan], np.float32)))


def test_sumsq_order_and_scale():
    rng = np.random.default_rng(5)
    x = (rng.standard_normal(50_000) * np.exp(rng.uniform(-20, 20, 50_000))).astype(np.float32)
    s = oracle.sumsq_f32(x)
    assert oracle.sumsq_f32(x[rng.permutation(x.size)]) == s  # exact, so order-free
    assert oracle.sumsq_f32(x * np.float32(2.0 ** 5)) == s * 2.0 ** 10


# --------------------------------------------------------------------------
# LAMB
# --------------------------------------------------------------------------

def _state(rng, n, grad_std=1e-3, scale=2.0 ** 12, warm=True):
    g = (rng.standard_normal(n) * grad_std * scale).astype(np.float32)
    g16 = g.astype(np.float16).view(np.uint16).copy()
    theta = (rng.standard_normal(n) * 0.02).astype(np.float32)
    if warm:
        m = (rng.standard_normal(n) * 1e-4).astype(np.float32)
        v = np.abs(rng.standard_normal(n) * 1e-6).astype(np.float32)
    else:
        m = np.zeros(n, np.float32)
        v = np.zeros(n, np.float32)
    return g16, theta, m, v, scale


def _run_lamb(g16, theta, m, v, seg, mult, lr, wd, t, phi_lo=0.0, phi_hi=math.inf):
    th, mm, vv = theta.copy(), m.copy(), v.copy()
    p16 = np.zeros(th.size, np.uint16)
    hp = oracle.hyper(lr, HP["beta1"], HP["beta2"], HP["eps"], wd, t)
    out = oracle.lamb(g16, th, mm, vv, p16, np.asarray(seg, np.int64), mult, hp, lr, phi_lo, phi_hi)
    return th, mm, vv, p16, out


def _run_adam(g16, theta, m, v, mult, lr, wd, t):
    th, mm, vv = theta.copy(), m.copy(), v.copy()
    p16 = np.zeros(th.size, np.uint16)
    oracle.adam(g16, th, mm, vv, p16, mult, oracle.hyper(lr, HP["beta1"], HP["beta2"], HP["eps"], wd, t))
    return th, mm, vv, p16


SEGS = [0, 1, 2, 5, 64, 1000, 1001, 4096, 5000]


@pytest.mark.parametrize("wd", [0.0, 0.01])
def test_lamb_moments_are_adams(wd):
    rng = np.random.default_rng(1)
    g16, theta, m, v, scale = _state(rng, SEGS[-1])
    mult = np.float32(1.0 / scale)
    _, m_l, v_l, _, _ = _run_lamb(g16, theta, m, v, SEGS, mult, 1e-3, wd, 7)
    _, m_a, v_a, _ = _run_adam(g16, theta, m, v, mult, 1e-3, wd, 7)
    assert np.array_equal(m_l.view(np.uint32), m_a.view(np.uint32))
    assert np.array_equal(v_l.view(np.uint32), v_a.view(np.uint32))


@pytest.mark.parametrize("wd", [0.0, 0.05])
def test_lamb_layer_update_norm_is_lr_times_weight_norm(wd):
    rng = np.random.default_rng(2)
    g16, theta, m, v, scale = _state(rng, SEGS[-1])
    lr = 0.1
    th, *_ , out = _run_lamb(g16, theta, m, v, SEGS, np.float32(1.0 / scale), lr, wd, 3)
    for s in range(len(SEGS) - 1):
        a, b = SEGS[s], SEGS[s + 1]
        w = np.linalg.norm(theta[a:b].astype(np.float64))
        d = np.linalg.norm(th[a:b].astype(np.float64) - theta[a:b].astype(np.float64))
        assert d == pytest.approx(lr * w, rel=2e-5), s
        assert out[s, 0] == pytest.approx(w * w, rel=1e-15)


@pytest.mark.parametrize("lo,hi,target", [(0.0, 1e-3, 1e-3), (10.0, math.inf, 10.0), (0.5, 0.5, 0.5)])
def test_lamb_phi_clamps_the_weight_norm(lo, hi, target):
    rng = np.random.default_rng(3)
    g16, theta, m, v, scale = _state(rng, 3000)
    lr = 0.1
    th, *_ = _run_lamb(g16, theta, m, v, [0, 3000], np.float32(1.0 / scale), lr, 0.0, 2, lo, hi)
    d = np.linalg.norm(th.astype(np.float64) - theta.astype(np.float64))
    assert d == pytest.approx(lr * target, rel=2e-5)


@pytest.mark.parametrize("k", [-3, 2, 9])
def test_lamb_is_invariant_to_rescaling_a_layer(k):
    # Without weight decay u does not depend on theta; scaling theta by 2^k scales the
    # trust ratio and so the update by exactly 2^k.
    rng = np.random.default_rng(4)
    g16, theta, m, v, scale = _state(rng, SEGS[-1])
    c = np.float32(2.0 ** k)
    mult = np.float32(1.0 / scale)
    th1, m1, v1, _, _ = _run_lamb(g16, theta, m, v, SEGS, mult, 1e-2, 0.0, 5)
    th2, m2, v2, _, _ = _run_lamb(g16, theta * c, m, v, SEGS, mult, 1e-2, 0.0, 5)
    assert np.array_equal((th1 * c).view(np.uint32), th2.view(np.uint32))
    assert np.array_equal(m1.view(np.uint32), m2.view(np.uint32)) and np.array_equal(v1.view(np.uint32),
                                                                                     v2.view(np.uint32))


@pytest.mark.parametrize("wd", [0.0, 0.01])
def test_lamb_zero_layer_takes_adams_step(wd):
    # ||theta|| = 0 gives trust ratio 1, so the step is lr*u: Adam's (decoupled decay of 0 adds 0)
    rng = np.random.default_rng(6)
    g16, _, m, v, scale = _state(rng, 4000)
    theta = np.zeros(4000, np.float32)
    mult = np.float32(1.0 / scale)
    th_l, m_l, v_l, p_l, out = _run_lamb(g16, theta, m, v, [0, 4000], mult, 1e-3, wd, 4)
    th_a, m_a, v_a, p_a = _run_adam(g16, theta, m, v, mult, 1e-3, wd, 4)
    assert out[0, 2] == 1.0
    for a, b in ((th_l, th_a), (m_l, m_a), (v_l, v_a)):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    assert np.array_equal(p_l, p_a)


def test_lamb_zero_update_leaves_layer_unchanged():
    n = 500
    theta = np.linspace(-1, 1, n).astype(np.float32)
    z = np.zeros(n, np.float32)
    th, m, v, _, out = _run_lamb(np.zeros(n, np.uint16), theta, z, z, [0, n], np.float32(1.0), 0.5, 0.0, 1)
    assert np.array_equal(th.view(np.uint32), theta.view(np.uint32)) and out[0, 1] == 0.0 and out[0, 2] == 1.0


@pytest.mark.parametrize("lr,wd", [(0.1, 0.01), (0.25, 0.5)])
def test_lamb_zero_gradient_with_decay_shrinks_by_one_minus_lr(lr, wd):
    # g = 0, m = v = 0: u = wd*theta, trust = ||theta||/(wd*||theta||), so theta <- (1-lr)*theta
    n = 777
    rng = np.random.default_rng(8)
    theta = (rng.standard_normal(n) * 0.5).astype(np.float32)
    z = np.zeros(n, np.float32)
    th, *_ = _run_lamb(np.zeros(n, np.uint16), theta, z, z, [0, n], np.float32(1.0), lr, wd, 1)
    want = theta.astype(np.float64) * (1 - lr)
    assert np.all(np.abs(th - want) <= 4 * np.spacing(np.abs(want).astype(np.float32)))


@pytest.mark.parametrize("theta0,g", [(2.0, 0.5), (-2.0, 0.5), (3.0, -0.25)])
def test_lamb_single_element_layer_moves_by_lr_times_weight(theta0, g):
    # One element per layer, first step from zero moments: u = g/(|g| + eps) ~ sign(g),
    # so the weight moves by lr*|theta| against the gradient.
    lr = 0.25
    g16 = np.array([g], np.float16).view(np.uint16)
    th, *_ = _run_lamb(g16, np.array([theta0], np.float32), np.zeros(1, np.float32), np.zeros(1, np.float32),
                       [0, 1], np.float32(1.0), lr, 0.0, 1)
    want = theta0 - math.copysign(lr * abs(theta0), g)
    assert abs(float(th[0]) - want) <= 2 * abs(float(np.spacing(np.float32(want))))


def test_lamb_layers_are_independent():
    rng = np.random.default_rng(9)
    g16, theta, m, v, scale = _state(rng, SEGS[-1])
    mult = np.float32(1.0 / scale)
    whole = _run_lamb(g16, theta, m, v, SEGS, mult, 1e-2, 0.01, 2)
    for s in range(len(SEGS) - 1):
        a, b = SEGS[s], SEGS[s + 1]
        one = _run_lamb(g16[a:b].copy(), theta[a:b].copy(), m[a:b].copy(), v[a:b].copy(), [0, b - a], mult, 1e-2,
                        0.01, 2)
        for x, y in zip(whole[:3], one[:3]):
            assert np.array_equal(x[a:b].view(np.uint32), y.view(np.uint32)), s
        assert np.array_equal(whole[3][a:b], one[3])
    # perturbing one layer changes nothing elsewhere
    theta2 = theta.copy()
    theta2[1001:4096] *= np.float32(3.0)
    other = _run_lamb(g16, theta2, m, v, SEGS, mult, 1e-2, 0.01, 2)
    keep = np.r_[0:1001, 4096:SEGS[-1]]
    assert np.array_equal(whole[0][keep].view(np.uint32), other[0][keep].view(np.uint32))


def test_lamb_fp16_copy_is_the_rounded_master():
    rng = np.random.default_rng(10)
    g16, theta, m, v, scale = _state(rng, 3000)
    th, _, _, p16, _ = _run_lamb(g16, theta, m, v, [0, 1000, 3000], np.float32(1.0 / scale), 1e-3, 0.0, 1)
    assert np.array_equal(p16, th.astype(np.float16).view(np.uint16))


def test_lamb_step_skips_on_overflow_and_rejects_bad_tables():
    rng = np.random.default_rng(12)
    g16, theta, m, v, scale = _state(rng, 100)
    g16[37] = 0x7C00
    th, mm, vv, p16 = theta.copy(), m.copy(), v.copy(), np.full(100, 0x1234, np.uint16)
    skip, sc, _ = oracle.lamb_step(g16, th, mm, vv, p16, [0, 50, 100], 1e-3, 0.9, 0.999, 1e-8, 0.0, 1, scale, 1.0)
    assert skip == 1 and sc.skip == 1
    assert np.array_equal(th, theta) and np.array_equal(mm, m) and np.array_equal(vv, v) and np.all(p16 == 0x1234)
    g16[37] = 0
    for bad in ([0, 50], [1, 100], [0, 50, 50, 100], [0, 60, 50, 100]):
        with pytest.raises(ValueError):
            oracle.lamb_step(g16, th, mm, vv, p16, bad, 1e-3, 0.9, 0.999, 1e-8, 0.0, 1, scale, 1.0)


def test_lamb_step_applies_the_clipped_gradient():
    # lamb_step = the Adam path's statistics and scalars, then zo_lamb with that multiplier
    rng = np.random.default_rng(13)
    g16, theta, m, v, scale = _state(rng, 2000, grad_std=5e-2)
    seg = [0, 700, 2000]
    a = [theta.copy(), m.copy(), v.copy(), np.zeros(2000, np.uint16)]
    skip, sc, out = oracle.lamb_step(g16, *a, seg, 1e-2, 0.9, 0.999, 1e-8, 0.0, 3, scale, 0.5)
    assert skip == 0 and sc.coef < 1.0  # the norm exceeds the clip: the multiplier carries the coefficient
    b = _run_lamb(g16, theta, m, v, seg, np.float32(sc.mult), 1e-2, 0.0, 3)
    for x, y in zip(a[:3], b[:3]):
        assert np.array_equal(x.view(np.uint32), y.view(np.uint32))
    assert np.array_equal(out, b[4])
