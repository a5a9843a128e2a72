"""Pins of the oracle's gradient statistics (ZeRO Sec. 3.2's gradient-norm pass
over the flattened gradients), the overflow test of loss-scaled mixed precision
and global-norm clipping.

The exact sum of squares is checked by brute force with Python fractions; the
norm by its closed form for constant gradients; the overflow test over every
non-finite binary16 pattern; the integer-to-double rounding against Python's
correctly rounded int -> float.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_1910_02054_amd import workloads


def _brute_force_units(g16: np.ndarray) -> int:
    total = Fraction(0)
    for b in g16.tolist():
        x = float(np.uint16(b).view(np.float16))
        if math.isfinite(x):
            total += Fraction(x) ** 2
    units = total * (1 << 48)
    assert units.denominator == 1
    return int(units)


@pytest.mark.parametrize("seed", range(6))
def test_exact_sum_matches_fractions(seed):
    r = np.random.default_rng(seed)
    n = int(r.integers(1, 3000))
    g16 = r.integers(0, 1 << 16, size=n, dtype=np.uint32).astype(np.uint16)
    g16 = g16[(g16 & 0x7C00) != 0x7C00]  # finite only; every exponent, subnormals, +-0
    g16 = np.concatenate([g16, np.array([0x7BFF, 0xFBFF, 0x0001, 0x8001, 0x0000, 0x8000], np.uint16)])
    s, ovf = oracle.local_stats(g16)
    assert ovf == 0
    assert s == _brute_force_units(g16)


def test_exact_sum_extreme_magnitudes():
    # n copies of +-65504: each k = 2047 * 2^29, so the sum needs about 80 + log2(n) bits.
    g16 = np.array([0x7BFF, 0xFBFF] * 5000, np.uint16)
    s, _ = oracle.local_stats(g16)
    assert s == 10000 * (2047 << 29) ** 2


@pytest.mark.parametrize("h", [0x3C00, 0x0001, 0x7BFF, 0xB555, 0x0400])
def test_constant_gradient_norm_closed_form(h):
    # norm of n equal values g is |g| * sqrt(n)
    n = 4096
    g16 = np.full(n, h, np.uint16)
    s, _ = oracle.local_stats(g16)
    sc = oracle.scalars(s, 0, 1.0, 0.0)
    g = abs(float(np.uint16(h).view(np.float16)))
    assert sc.norm == g * math.sqrt(n)


def test_sum_is_additive_across_partitions():
    g16, *_ = workloads.random_case(3, 100_003)
    whole, _ = oracle.local_stats(g16)
    parts = sum(oracle.local_stats(g16[a:a + 7919])[0] for a in range(0, g16.size, 7919))
    assert parts == whole


def test_every_nonfinite_pattern_is_overflow():
    base = np.full(17, 0x3C00, np.uint16)
    nonfinite = [e | f | s for s in (0, 0x8000) for e in (0x7C00,) for f in range(0, 1024)]
    for pos in (0, 8, 16):
        for h in nonfinite[::37] + [0x7C00, 0xFC00, 0x7E00, 0x7C01, 0xFFFF]:
            g = base.copy()
            g[pos] = h
            assert oracle.local_stats(g)[1] == 1, hex(h)


def test_largest_finite_values_are_not_overflow():
    g = np.array([0x7BFF, 0xFBFF, 0x0000, 0x8000, 0x03FF], np.uint16)
    assert oracle.local_stats(g)[1] == 0


def test_lone_inf_in_last_element():
    g16, *_ = workloads.random_case(5, 12_345)
    g16[-1] = 0x7C00
    assert oracle.local_stats(g16)[1] == 1
    g16[-1] = 0x3C00
    g16[0] = 0x7E01
    assert oracle.local_stats(g16)[1] == 1


def test_u128_to_double_rounds_to_nearest_even():
    r = np.random.default_rng(1)
    vals = [int(x) for x in r.integers(0, 1 << 63, size=200, dtype=np.uint64)]
    vals = [(a << 64 | b) >> int(s) for a, b, s in zip(vals, vals[::-1], r.integers(0, 60, size=200))]
    vals += [(1 << 53) + 1, (1 << 54) + 2, (1 << 54) + 6, (1 << 108) - 1, (1 << 127) + (1 << 74), 0, 1]
    for v in vals:
        assert oracle.u128_to_double(v) == float(v), v


def test_clip_coefficient_cases():
    one = 1 << 48  # one unit of g^2 = 1.0 in units of 2^-48
    # norm == clip: not clipped (strict comparison)
    sc = oracle.scalars(one, 0, 1.0, 1.0)
    assert (sc.norm, sc.coef) == (1.0, 1.0)
    # clip <= 0 disables clipping
    assert oracle.scalars(100 * one, 0, 1.0, 0.0).coef == 1.0
    assert oracle.scalars(100 * one, 0, 1.0, -1.0).coef == 1.0
    # norm 10 > clip 1: coefficient 0.1 and the clipped norm equals clip
    sc = oracle.scalars(100 * one, 0, 1.0, 1.0)
    assert sc.norm == 10.0 and sc.coef * sc.norm == pytest.approx(1.0, rel=2 ** -52)
    # the loss scale is divided out of the norm: sum g16^2 = 2^32 * 100 at scale 2^16 -> norm 10
    sc = oracle.scalars(100 * one << 32, 0, 2.0 ** 16, 0.0)
    assert sc.norm == 10.0 and sc.mult == np.float32(2.0 ** -16)
    # with clipping the multiplier folds both: coef / scale
    sc = oracle.scalars(100 * one << 32, 0, 2.0 ** 16, 1.0)
    assert sc.mult == np.float32(0.1 / 2.0 ** 16)


def test_overflow_sets_skip():
    sc = oracle.scalars(0, 1, 2.0 ** 16, 1.0)
    assert sc.skip == 1
    assert oracle.scalars(0, 0, 2.0 ** 16, 1.0).skip == 0
