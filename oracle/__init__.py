"""CPU oracle of the ZeRO P_os+g shard optimizer step -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It never touches the GPU library and
the GPU library never touches it; the only code both sides share is the seeded
input generator module, which holds none of the method's arithmetic.

Two independent implementations live here:

* ``zero_oracle.c`` (loaded below through ctypes): scalar C, exact integer sum
  of squares, binary16 coding from the format definition, fp32 Adam.
* ``twin.py``: the same specification written again in numpy, used to
  cross-check the C oracle bit for bit on small inputs.

Every function cites the passage of ZeRO (arXiv 1910.02054) or of the method
it cites that it follows; see ``zero_oracle.c``'s header.
"""
import ctypes
import os
import threading

import numpy as np

from . import build as _build

_lib = None
_lock = threading.Lock()


class Scalars(ctypes.Structure):
    _fields_ = [("sumsq", ctypes.c_double), ("norm", ctypes.c_double), ("coef", ctypes.c_double),
                ("mult", ctypes.c_float), ("skip", ctypes.c_int32)]


class Hyper(ctypes.Structure):
    _fields_ = [(k, ctypes.c_float) for k in ("lr", "b1", "omb1", "b2", "omb2", "bc1", "bc2", "eps", "wd")]


def lib():
    """Load the oracle library, compiling it first when it is not built."""
    global _lib
    with _lock:
        if _lib is None:
            # ZERO_ORACLE_LIB points the pin suite at a deliberately mutated build (mutation tests).
            path = os.environ.get("ZERO_ORACLE_LIB")
            if not path:
                path = _build.LIB
                if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_build.SRC):
                    _build.build()
            L = ctypes.CDLL(path)
            P = ctypes.c_void_p
            i64, i32, dbl, flt = ctypes.c_int64, ctypes.c_int32, ctypes.c_double, ctypes.c_float
            L.zo_layout.argtypes = [i64, i32, i32, P]
            L.zo_layout.restype = ctypes.c_int
            L.zo_f16_to_f32.argtypes = [ctypes.c_uint16]
            L.zo_f16_to_f32.restype = flt
            L.zo_f32_to_f16.argtypes = [flt]
            L.zo_f32_to_f16.restype = ctypes.c_uint16
            L.zo_f32_to_f16_array.argtypes = [P, P, i64]
            L.zo_f32_to_f16_array.restype = None
            L.zo_local_stats.argtypes = [P, i64, P, P]
            L.zo_local_stats.restype = None
            L.zo_u128_to_double.argtypes = [P]
            L.zo_u128_to_double.restype = dbl
            L.zo_scalars.argtypes = [P, i32, dbl, dbl, ctypes.POINTER(Scalars)]
            L.zo_scalars.restype = None
            L.zo_hyper.argtypes = [dbl, dbl, dbl, dbl, dbl, i64, ctypes.POINTER(Hyper)]
            L.zo_hyper.restype = None
            L.zo_adam.argtypes = [P, P, P, P, P, i64, flt, ctypes.POINTER(Hyper)]
            L.zo_adam.restype = None
            L.zo_shard_step.argtypes = [P, P, P, P, P, i64, dbl, dbl, dbl, dbl, dbl, i64, dbl, dbl,
                                        ctypes.POINTER(Scalars)]
            L.zo_shard_step.restype = ctypes.c_int
            L.zo_model_state_bytes.argtypes = [dbl, dbl, i32, dbl]
            L.zo_model_state_bytes.restype = dbl
            L.zo_scaler_update.argtypes = [ctypes.POINTER(dbl), ctypes.POINTER(i64), ctypes.POINTER(i64), i32,
                                           i64, dbl]
            L.zo_scaler_update.restype = None
            L.zo_sumsq_f32.argtypes = [P, i64]
            L.zo_sumsq_f32.restype = dbl
            L.zo_lamb.argtypes = [P, P, P, P, P, i64, P, i32, flt, ctypes.POINTER(Hyper), dbl, dbl, dbl, P]
            L.zo_lamb.restype = ctypes.c_int
            L.zo_lamb_step.argtypes = [P, P, P, P, P, i64, P, i32, dbl, dbl, dbl, dbl, dbl, i64, dbl, dbl, dbl,
                                       dbl, ctypes.POINTER(Scalars), P]
            L.zo_lamb_step.restype = ctypes.c_int
            _lib = L
    return _lib


def _ptr(a: np.ndarray, dtype) -> int:
    if a.dtype != dtype or not a.flags.c_contiguous:
        raise TypeError("expected a C-contiguous %s array, got %s" % (np.dtype(dtype), a.dtype))
    return a.ctypes.data


# --------------------------------------------------------------------------
# Layout (Sec. 5.1)
# --------------------------------------------------------------------------

def layout(psi: int, nd: int, rank: int):
    """(S, offset, valid, padded_total) of rank's shard; Sec. 5.1 equal partitions,
    tail-padded when N_d does not divide Psi.  Raises ValueError on bad input."""
    out = (ctypes.c_int64 * 4)()
    if lib().zo_layout(psi, nd, rank, out) != 0:
        raise ValueError("invalid layout arguments psi=%r nd=%r rank=%r" % (psi, nd, rank))
    return tuple(int(x) for x in out)


# --------------------------------------------------------------------------
# binary16 coding
# --------------------------------------------------------------------------

def f16_to_f32(h: int) -> float:
    return float(lib().zo_f16_to_f32(h))


def f32_to_f16(x: float) -> int:
    return int(lib().zo_f32_to_f16(x))


def f32_to_f16_array(x: np.ndarray) -> np.ndarray:
    """Element-wise binary16 encoding (uint16 bit patterns) of a float32 array."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.size, np.uint16)
    lib().zo_f32_to_f16_array(_ptr(x, np.float32), _ptr(out, np.uint16), x.size)
    return out


# --------------------------------------------------------------------------
# Statistics and scalars (Sec. 3.2 gradient norm; loss scaling; clipping)
# --------------------------------------------------------------------------

def local_stats(g16: np.ndarray):
    """(sum of k^2 as a Python int in units of 2^-48, overflow flag) of one shard."""
    g = np.ascontiguousarray(g16).view(np.uint16)
    s = (ctypes.c_uint64 * 2)()
    ovf = ctypes.c_int32()
    lib().zo_local_stats(_ptr(g, np.uint16), g.size, s, ctypes.byref(ovf))
    return int(s[0]) | (int(s[1]) << 64), int(ovf.value)


def u128_to_double(v: int) -> float:
    s = (ctypes.c_uint64 * 2)(v & ((1 << 64) - 1), v >> 64)
    return float(lib().zo_u128_to_double(s))


def scalars(sumsq_units: int, overflow: int, loss_scale: float, clip: float) -> Scalars:
    if not 0 <= sumsq_units < (1 << 128):
        raise ValueError("sum of squares out of the 128-bit range")
    s = (ctypes.c_uint64 * 2)(sumsq_units & ((1 << 64) - 1), sumsq_units >> 64)
    out = Scalars()
    lib().zo_scalars(s, overflow, loss_scale, clip, ctypes.byref(out))
    return out


def hyper(lr, beta1, beta2, eps, wd, t) -> Hyper:
    h = Hyper()
    lib().zo_hyper(lr, beta1, beta2, eps, wd, t, ctypes.byref(h))
    return h


# --------------------------------------------------------------------------
# The update (Adam, Kingma & Ba; mixed precision as in Sec. 3.1)
# --------------------------------------------------------------------------

def adam(g16, theta, m, v, p16, mult: float, hp: Hyper):
    """In-place fp32 Adam on numpy arrays (g16 and p16 as uint16 bit patterns)."""
    n = g16.size
    for a in (theta, m, v, p16):
        if a.size != n:
            raise ValueError("shard arrays differ in length")
    lib().zo_adam(_ptr(g16, np.uint16), _ptr(theta, np.float32), _ptr(m, np.float32), _ptr(v, np.float32),
                  _ptr(p16, np.uint16), n, mult, ctypes.byref(hp))


def shard_step(g16, theta, m, v, p16, lr, beta1, beta2, eps, wd, t, loss_scale, clip):
    """One whole step on numpy arrays, in place.  Returns (skipped, Scalars)."""
    n = g16.size
    for a in (theta, m, v, p16):
        if a.size != n:
            raise ValueError("shard arrays differ in length")
    sc = Scalars()
    r = lib().zo_shard_step(_ptr(g16, np.uint16), _ptr(theta, np.float32), _ptr(m, np.float32),
                            _ptr(v, np.float32), _ptr(p16, np.uint16), n, lr, beta1, beta2, eps, wd, t,
                            loss_scale, clip, ctypes.byref(sc))
    return int(r), sc


# --------------------------------------------------------------------------
# LAMB (You et al.; listed by ZeRO's related work among the adaptive optimizers
# whose memory ZeRO reduces)
# --------------------------------------------------------------------------

def sumsq_f32(x: np.ndarray) -> float:
    """Exact sum of squares of a float32 array, rounded once to double."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    return float(lib().zo_sumsq_f32(_ptr(x, np.float32), x.size))


def _segments(seg_off, n):
    off = np.ascontiguousarray(seg_off, dtype=np.int64)
    if off.ndim != 1 or off.size < 1:
        raise ValueError("seg_off must be a 1-D array of n_seg + 1 offsets")
    return off, off.size - 1


def lamb(g16, theta, m, v, p16, seg_off, mult: float, hp: Hyper, lr: float, phi_lo: float = 0.0,
         phi_hi: float = float("inf")):
    """In-place LAMB update on numpy arrays; returns an (n_seg, 3) array of
    (sum theta^2, sum u^2, trust ratio) per layer."""
    n = g16.size
    for a in (theta, m, v, p16):
        if a.size != n:
            raise ValueError("shard arrays differ in length")
    off, n_seg = _segments(seg_off, n)
    out = np.empty((max(n_seg, 1), 3), np.float64)
    r = lib().zo_lamb(_ptr(g16, np.uint16), _ptr(theta, np.float32), _ptr(m, np.float32), _ptr(v, np.float32),
                      _ptr(p16, np.uint16), n, off.ctypes.data, n_seg, mult, ctypes.byref(hp), lr, phi_lo, phi_hi,
                      out.ctypes.data)
    if r != 0:
        raise ValueError("malformed layer table")
    return out[:n_seg]


def lamb_step(g16, theta, m, v, p16, seg_off, lr, beta1, beta2, eps, wd, t, loss_scale, clip, phi_lo=0.0,
              phi_hi=float("inf")):
    """One whole LAMB step in place.  Returns (skipped, Scalars, per-layer array)."""
    n = g16.size
    for a in (theta, m, v, p16):
        if a.size != n:
            raise ValueError("shard arrays differ in length")
    off, n_seg = _segments(seg_off, n)
    out = np.zeros((max(n_seg, 1), 3), np.float64)
    sc = Scalars()
    r = lib().zo_lamb_step(_ptr(g16, np.uint16), _ptr(theta, np.float32), _ptr(m, np.float32), _ptr(v, np.float32),
                           _ptr(p16, np.uint16), n, off.ctypes.data, n_seg, lr, beta1, beta2, eps, wd, t, loss_scale,
                           clip, phi_lo, phi_hi, ctypes.byref(sc), out.ctypes.data)
    if r < 0:
        raise ValueError("malformed layer table")
    return int(r), sc, out[:n_seg]


# --------------------------------------------------------------------------
# Memory accounting (Sec. 3.1, Sec. 5.1-5.3) and loss scaling
# --------------------------------------------------------------------------

STAGE_DP, STAGE_OS, STAGE_OS_G, STAGE_OS_G_P = 0, 1, 2, 3


def model_state_bytes(psi: float, nd: float, stage: int, k: float = 12.0) -> float:
    r = lib().zo_model_state_bytes(psi, nd, stage, k)
    if r < 0:
        raise ValueError("bad stage or N_d")
    return float(r)


class Scaler:
    """Dynamic loss-scale state driven by the oracle's update rule."""

    def __init__(self, scale: float, window: int = 1000, min_scale: float = 1.0):
        self.scale = ctypes.c_double(scale)
        self.applied = ctypes.c_int64(0)
        self.good = ctypes.c_int64(0)
        self.window = window
        self.min_scale = min_scale

    @property
    def t_next(self) -> int:
        """Adam's 1-based t for the next applied update."""
        return self.applied.value + 1

    def update(self, skipped: bool):
        lib().zo_scaler_update(ctypes.byref(self.scale), ctypes.byref(self.applied), ctypes.byref(self.good),
                               1 if skipped else 0, self.window, self.min_scale)
