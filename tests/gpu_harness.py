"""Helpers shared by the GPU parity tests and the smoke check: guarded device
buffers, a thread-parallel driver of the CPU oracle, and the parity comparison.

The oracle is run chunk by chunk in threads (ctypes releases the GIL): exact
per-chunk sums of squares are added as integers and the element-wise update is
applied per chunk with the combined scalars.  That this equals one
unpartitioned oracle call bit for bit is the partition-invariance pin in
tests/test_oracle_invariants.py.
"""
import os
import sys
from concurrent.futures import ThreadPoolExecutor

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402

GUARD = 1024          # guard elements on each side of every device buffer
GUARD_BYTE = 0xA5
_CHUNK = 1 << 22


def _workers():
    try:
        return max(1, min(16, len(os.sched_getaffinity(0))))
    except AttributeError:
        return 4


_POOL = ThreadPoolExecutor(max_workers=_workers())


def oracle_step(g16, theta, m, v, p16, lr, beta1, beta2, eps, wd, t, scale, clip):
    """In-place oracle step over host arrays; returns (skip, Scalars)."""
    n = g16.size
    spans = [(a, min(n, a + _CHUNK)) for a in range(0, n, _CHUNK)]
    parts = list(_POOL.map(lambda s: oracle.local_stats(g16[s[0]:s[1]]), spans))
    total = sum(p[0] for p in parts)
    ovf = 1 if any(p[1] for p in parts) else 0
    sc = oracle.scalars(total, ovf, scale, clip)
    if sc.skip:
        return 1, sc
    hp = oracle.hyper(lr, beta1, beta2, eps, wd, t)

    def upd(s):
        a, b = s
        oracle.adam(g16[a:b], theta[a:b], m[a:b], v[a:b], p16[a:b], sc.mult, hp)

    list(_POOL.map(upd, spans))
    return 0, sc


def oracle_lamb_step(g16, theta, m, v, p16, seg_off, lr, beta1, beta2, eps, wd, t, scale, clip, phi_lo=0.0,
                     phi_hi=float("inf"), global_sumsq_units=None):
    """In-place oracle LAMB step over host arrays; returns (skip, Scalars, per-layer array).

    The gradient statistics are exact per chunk (threads); the layers are then
    updated one oracle call each, in threads (layers are independent given the
    multiplier: pinned in tests/test_oracle_lamb.py).  global_sumsq_units
    replaces the local statistics (the split-phase case: the sum over every
    rank's gradient)."""
    n = g16.size
    if global_sumsq_units is None:
        spans = [(a, min(n, a + _CHUNK)) for a in range(0, n, _CHUNK)]
        parts = list(_POOL.map(lambda s: oracle.local_stats(g16[s[0]:s[1]]), spans))
        total, ovf = sum(p[0] for p in parts), (1 if any(p[1] for p in parts) else 0)
    else:
        total, ovf = global_sumsq_units
    sc = oracle.scalars(total, ovf, scale, clip)
    if sc.skip:
        return 1, sc, None
    hp = oracle.hyper(lr, beta1, beta2, eps, wd, t)
    off = np.asarray(seg_off, np.int64)

    def run(k):
        a, b = int(off[k]), int(off[k + 1])
        return oracle.lamb(g16[a:b], theta[a:b], m[a:b], v[a:b], p16[a:b], np.array([0, b - a], np.int64),
                           sc.mult, hp, lr, phi_lo, phi_hi)

    outs = list(_POOL.map(run, range(off.size - 1)))
    return 0, sc, np.concatenate(outs) if outs else np.zeros((0, 3))


class Guarded:
    """A device buffer of n elements with GUARD canary elements on both sides
    (and optional extra leading elements to misalign the view)."""

    def __init__(self, torch, n, dtype, device, shift=0):
        self.torch = torch
        self.n, self.shift = n, shift
        self.buf = torch.empty(n + 2 * GUARD + shift, dtype=dtype, device=device)
        self.buf.view(torch.uint8).fill_(GUARD_BYTE)
        self.view = self.buf[GUARD + shift:GUARD + shift + n]
        self.host = None

    def guards_intact(self):
        t = self.torch
        raw = self.buf.view(t.uint8)
        es = self.buf.element_size()
        lo = raw[:(GUARD + self.shift) * es]
        hi = raw[(GUARD + self.shift + self.n) * es:]
        return bool((lo == GUARD_BYTE).all().item()) and bool((hi == GUARD_BYTE).all().item())

    def upload(self, arr):
        t = self.torch
        a = np.ascontiguousarray(arr)
        if self.buf.dtype == t.float16:
            src = t.from_numpy(a.view(np.int16)).view(t.float16)
        else:
            src = t.from_numpy(a)
        self.view.copy_(src)

    def download(self):
        """The view's contents as a numpy array backed by a reused pinned host buffer
        (overwritten by the next download: copy it to keep it)."""
        t = self.torch
        if self.host is None:
            self.host = t.empty(self.n, dtype=self.buf.dtype, pin_memory=True)
        self.host.copy_(self.view)
        x = self.host.view(t.int16) if self.buf.dtype == t.float16 else self.host
        return x.numpy().view(np.uint16 if x.dtype == t.int16 else np.float32)


def ulp_distance16(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """|a - b| in binary16 ulps, comparing sign-magnitude bit patterns as ordered integers."""
    def key(x):
        x = x.astype(np.int32)
        return np.where(x & 0x8000, -(x & 0x7FFF), x & 0x7FFF)
    return np.abs(key(a) - key(b))


def _mismatches(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Indices where the bit patterns of a and b differ (chunked over threads)."""
    n = a.size
    spans = [(s, min(n, s + _CHUNK)) for s in range(0, n, _CHUNK)]
    parts = list(_POOL.map(lambda s: s[0] + np.flatnonzero(a[s[0]:s[1]] != b[s[0]:s[1]]), spans))
    return np.concatenate(parts) if parts else np.empty(0, np.int64)


def compare_state(gpu, ref, tol=1e-6):
    """Parity of (theta, m, v, p16): returns a dict of diagnostics; raises AssertionError
    when master/m/v exceed max|d| <= tol*max(1,|x_oracle|) or p16 differs by > 1 ulp."""
    out = {}
    for name, g, r in zip(("master", "m", "v"), gpu[:3], ref[:3]):
        idx = _mismatches(g.view(np.uint32), r.view(np.uint32))
        nbad = int(idx.size)
        out[name + "_bitdiff"] = nbad
        if nbad:
            gd, rd = g[idx].astype(np.float64), r[idx].astype(np.float64)
            err = np.abs(gd - rd)
            lim = tol * np.maximum(1.0, np.abs(rd))
            assert np.all(np.isfinite(gd)), "%s: non-finite GPU values" % name
            worst = int(np.argmax(err / lim))
            assert np.all(err <= lim), "%s: |d|=%g > %g at %d" % (name, err[worst], lim[worst], idx[worst])
            rel = err / np.maximum(np.abs(rd), 1e-30)
            out[name + "_max_abs"] = float(err.max())
            out[name + "_max_rel"] = float(rel.max())
    idx = _mismatches(gpu[3], ref[3])
    nbad = int(idx.size)
    out["p16_bitdiff"] = nbad
    if nbad:
        d = ulp_distance16(gpu[3][idx], ref[3][idx])
        assert d.max() <= 1, "p16 off by %d ulp at %d" % (int(d.max()), int(idx[int(np.argmax(d))]))
    return out
