"""Numpy twin of the C oracle -- TEST INFRASTRUCTURE.

A second, independently written implementation of the same step, used only to
cross-check ``zero_oracle.c`` bit for bit on small inputs.  Where the C oracle
decodes and encodes binary16 from the format definition and sums squares in a
128-bit integer, this twin lets numpy's own float16 conversions do the coding
and sums squares with Python integers.  The fp32 update is the same sequence
of correctly rounded operations (Adam with bias correction, Kingma & Ba, the
optimizer ZeRO's Sec. 3.1 builds its K = 12 accounting on).
"""
import math

import numpy as np

_CHUNK = 1 << 22


def exact_sumsq_units(g16: np.ndarray):
    """(sum of (g * 2^24)^2 over finite elements as a Python int, overflow flag)."""
    h = np.ascontiguousarray(g16).view(np.float16)
    finite = np.isfinite(h)
    overflow = int(not bool(finite.all()))
    total = 0
    for s in range(0, h.size, _CHUNK):
        blk = h[s:s + _CHUNK][finite[s:s + _CHUNK]]
        # |g| * 2^24 is an integer below 2^40, exact in float64 and int64.
        k = np.abs(blk.astype(np.float64) * float(1 << 24)).astype(np.int64)
        hi, lo = k >> 20, k & ((1 << 20) - 1)
        # k^2 = hi^2 * 2^40 + 2*hi*lo * 2^20 + lo^2; each partial sum stays below 2^63.
        total += (int(np.sum(hi * hi)) << 40) + (int(np.sum(hi * lo)) << 21) + int(np.sum(lo * lo))
    return total, overflow


def scalars(sumsq_units: int, overflow: int, loss_scale: float, clip: float):
    """(skip, norm, coef, mult) -- clipping of the unscaled gradient's global norm."""
    if overflow:
        return 1, math.inf, 1.0, np.float32(0.0)
    sumsq = math.ldexp(float(sumsq_units), -48)  # int -> float rounds to nearest even
    norm = math.sqrt(sumsq) / loss_scale
    coef = clip / norm if (clip > 0.0 and norm > clip) else 1.0
    return 0, norm, coef, np.float32(coef / loss_scale)


def adam(g16, theta, m, v, mult, lr, beta1, beta2, eps, wd, t):
    """Returns new (theta, m, v, p16) as fresh arrays; inputs are not modified."""
    f = np.float32
    lr32, b1, omb1, b2, omb2 = f(lr), f(beta1), f(1.0 - beta1), f(beta2), f(1.0 - beta2)
    bc1, bc2, eps32, wd32 = f(1.0 - beta1 ** t), f(1.0 - beta2 ** t), f(eps), f(wd)
    g = np.ascontiguousarray(g16).view(np.float16).astype(np.float32) * f(mult)
    m2 = b1 * m + omb1 * g
    v2 = b2 * v + omb2 * (g * g)
    u = (m2 / bc1) / (np.sqrt(v2 / bc2) + eps32)
    if wd32 != 0:
        u = u + wd32 * theta
    th = theta - lr32 * u
    return th.astype(np.float32), m2, v2, th.astype(np.float16).view(np.uint16)


def shard_step(g16, theta, m, v, lr, beta1, beta2, eps, wd, t, loss_scale, clip):
    """Whole step; returns (skip, new_theta, new_m, new_v, p16 or None)."""
    s, ovf = exact_sumsq_units(g16)
    skip, _norm, _coef, mult = scalars(s, ovf, loss_scale, clip)
    if skip:
        return 1, theta.copy(), m.copy(), v.copy(), None
    th, m2, v2, p16 = adam(g16, theta, m, v, mult, lr, beta1, beta2, eps, wd, t)
    return 0, th, m2, v2, p16
