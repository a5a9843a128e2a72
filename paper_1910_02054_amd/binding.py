"""Thin ctypes binding of ``libzeroshard.so`` (C ABI in ``include/zero_shard.h``).

Argument marshalling only: every step of the path runs in the library's HIP
kernels.  PyTorch supplies device memory (``data_ptr()``) and streams.  There
is no fallback: if the library is not built, importing this module raises.
"""
import ctypes
import os

from . import build as _build

ZERO_OK, ZERO_SKIPPED, ZERO_EINVAL, ZERO_EHIP, ZERO_ENOMEM = 0, 1, -1, -2, -3
ZERO_STAGE_DP, ZERO_STAGE_OS, ZERO_STAGE_OS_G, ZERO_STAGE_OS_G_P = 0, 1, 2, 3

if not os.path.exists(_build.LIB):
    raise ImportError("libzeroshard.so is not built (%s); run __graft_entry__.build() or "
                      "python paper_1910_02054_amd/build.py" % _build.LIB)
_lib = ctypes.CDLL(_build.LIB)
LIB_PATH = _build.LIB


class ZeroError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__("%s (code %d)" % (msg, code))
        self.code = code


class Layout(ctypes.Structure):
    _fields_ = [("shard_numel", ctypes.c_int64), ("offset", ctypes.c_int64), ("valid_numel", ctypes.c_int64),
                ("padded_total", ctypes.c_int64)]


class StepStats(ctypes.Structure):
    _fields_ = [("sumsq", ctypes.c_double), ("norm", ctypes.c_double), ("coef", ctypes.c_double),
                ("mult", ctypes.c_float), ("overflow", ctypes.c_int32), ("skipped", ctypes.c_int32),
                ("path", ctypes.c_int32), ("n", ctypes.c_int64)]


class ScalerState(ctypes.Structure):
    _fields_ = [("scale", ctypes.c_double), ("min_scale", ctypes.c_double), ("window", ctypes.c_int64),
                ("applied", ctypes.c_int64), ("good", ctypes.c_int64)]


class StepArgs(ctypes.Structure):
    """Mirror of zero_step_args_t (the fixed arguments of a training loop's step)."""
    _fields_ = [(k, ctypes.c_void_p) for k in ("grad16", "master32", "m32", "v32", "param16_out")] + \
               [("n", ctypes.c_int64)] + \
               [(k, ctypes.c_double) for k in ("lr", "beta1", "beta2", "eps", "weight_decay", "clip")] + \
               [("stream", ctypes.c_void_p)]


class Profile(ctypes.Structure):
    _fields_ = [("steps", ctypes.c_int64), ("stats_ms", ctypes.c_double), ("update_ms", ctypes.c_double)]


class ResidentState(ctypes.Structure):
    """Mirror of zero_resident_state_t (the resident step's device record)."""
    _fields_ = [(k, ctypes.c_double) for k in ("lr", "beta1", "beta2", "eps", "weight_decay", "clip", "loss_scale",
                                               "min_scale")] + \
               [(k, ctypes.c_int64) for k in ("window", "t", "good", "steps")] + \
               [("skipped", ctypes.c_int32), ("pad_", ctypes.c_int32)]


class LambProfile(ctypes.Structure):
    _fields_ = [("steps", ctypes.c_int64), ("stats_ms", ctypes.c_double), ("moments_ms", ctypes.c_double),
                ("layer_ms", ctypes.c_double), ("apply_ms", ctypes.c_double)]


_P, _i64, _i32, _dbl = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_double
_lib.zero_partition_layout.argtypes = [_i64, _i32, _i32, ctypes.POINTER(Layout)]
_lib.zero_shard_step.argtypes = [_P, _P, _P, _P, _P, _i64, _dbl, _dbl, _dbl, _dbl, _dbl, _i64, _dbl, _dbl, _P]
_lib.zero_shard_stats.argtypes = [_P, _i64, ctypes.POINTER(_dbl), _P]
_lib.zero_shard_apply.argtypes = [_P, _P, _P, _P, _P, _i64, _dbl, _dbl, _dbl, _dbl, _dbl, _dbl, _i64, _dbl, _dbl, _P]
_lib.zero_shard_validate.argtypes = [_P, _P, _P, _P, _P, _i64]
_lib.zero_shard_last_stats.argtypes = [ctypes.POINTER(_dbl), ctypes.POINTER(ctypes.c_float),
                                       ctypes.POINTER(ctypes.c_int)]
_lib.zero_shard_last_step_stats.argtypes = [ctypes.POINTER(StepStats)]
_lib.zero_memory_bytes.argtypes = [_dbl, _i32, _i32, _i32, ctypes.POINTER(_dbl)]
_lib.zero_bias_corrections.argtypes = [_dbl, _dbl, _i64, ctypes.POINTER(ctypes.c_float),
                                       ctypes.POINTER(ctypes.c_float)]
_lib.zero_resident_state_init.argtypes = [_P, _dbl, _dbl, _dbl, _dbl, _dbl, _dbl, _dbl, _dbl, _i64, _i64]
_lib.zero_resident_release.argtypes = [_P]
_lib.zero_stream_release.argtypes = [_P]
_lib.zero_workspace_count.argtypes = [ctypes.POINTER(_i64), ctypes.POINTER(_i64)]
_lib.zero_probe_lamb_pass.argtypes = [_i32, _P, _P, _P, _P, _P, _i64, _P]
_lib.zero_probe_adam_mix.argtypes = [_P, _P, _P, _P, _P, _i64, _P]
_lib.zero_shard_step_scaled.argtypes = [_P, _P]
_lib.zero_shard_step_noalloc.argtypes = _lib.zero_shard_step.argtypes
_lib.zero_scaler_init.argtypes = [ctypes.POINTER(ScalerState), _dbl, _i64, _dbl]
_lib.zero_scaler_update.argtypes = [ctypes.POINTER(ScalerState), _i32]
_lib.zero_model_state_bytes.argtypes = [_dbl, _dbl, _i32, _dbl, ctypes.POINTER(_dbl)]
_lib.zero_last_error.argtypes = []
_lib.zero_last_error.restype = ctypes.c_char_p
_lib.zero_profile_enable.argtypes = [_i32]
_lib.zero_profile_read.argtypes = [ctypes.POINTER(Profile)]
_lib.zero_probe_copy.argtypes = [_P, _P, _i64, _P]
_lib.zero_shard_stats_async.argtypes = [_P, _i64, _P, _P]
_lib.zero_shard_apply_async.argtypes = [_P, _P, _P, _P, _P, _i64, _P, _dbl, _dbl, _dbl, _dbl, _dbl, _i64, _dbl, _dbl,
                                        _P, _P]
_lib.zero_shard_step_resident.argtypes = [_P, _P, _P, _P, _P, _i64, _P, _P]
_lib.zero_lamb_plan_create.argtypes = [_P, _i32, _i64, ctypes.POINTER(_P)]
_lib.zero_lamb_plan_destroy.argtypes = [_P]
_lib.zero_lamb_step.argtypes = [_P, _P, _P, _P, _P, _P, _dbl, _dbl, _dbl, _dbl, _dbl, _i64, _dbl, _dbl, _dbl, _dbl, _P]
_lib.zero_lamb_moments.argtypes = [_P, _P, _P, _P, _P, _dbl, _dbl, _dbl, _dbl, _dbl, _i64, _dbl, _dbl, _P, _P]
_lib.zero_lamb_apply.argtypes = [_P, _P, _P, _P, _P, _dbl, _P, _dbl, _dbl, _dbl, _dbl, _dbl, _i64, _dbl, _dbl, _P]
_lib.zero_lamb_profile_read.argtypes = [ctypes.POINTER(LambProfile)]
EXPORTS = ("zero_partition_layout", "zero_shard_step", "zero_shard_stats", "zero_shard_apply",
           "zero_shard_validate", "zero_shard_last_stats", "zero_shard_last_step_stats", "zero_scaler_init",
           "zero_scaler_update", "zero_memory_bytes", "zero_model_state_bytes", "zero_bias_corrections",
           "zero_last_error", "zero_profile_enable", "zero_profile_read", "zero_probe_copy",
           "zero_lamb_plan_create", "zero_lamb_plan_destroy", "zero_lamb_step", "zero_lamb_moments",
           "zero_lamb_apply", "zero_lamb_profile_read", "zero_shard_stats_async", "zero_shard_apply_async",
           "zero_resident_state_init", "zero_shard_step_resident", "zero_resident_release",
           "zero_stream_release", "zero_workspace_count", "zero_probe_lamb_pass", "zero_shard_step_noalloc",
           "zero_probe_adam_mix", "zero_shard_step_scaled")
for _f in EXPORTS:
    if _f != "zero_last_error":
        getattr(_lib, _f).restype = ctypes.c_int


def _check(rc):
    if rc < 0:
        raise ZeroError(rc, _lib.zero_last_error().decode(errors="replace"))
    return rc


def _addr(x, dtypes=None, what="array"):
    """Device address of a torch tensor (checked) or a raw integer address."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if dtypes is not None and x.dtype not in dtypes:
        raise TypeError("%s: dtype %s not in %s" % (what, x.dtype, dtypes))
    if not x.is_cuda:
        raise TypeError("%s must be a device tensor" % what)
    if not x.is_contiguous():
        raise TypeError("%s must be contiguous" % what)
    return x.data_ptr()


def _shard_len(n, *arrays):
    """The element count of a shard call.  With n None: the common length of the tensors
    (all arguments must be tensors).  An explicit n may not exceed any tensor's length;
    for raw integer addresses the caller vouches for the size."""
    ts = [a for a in arrays if a is not None and not isinstance(a, int)]
    if n is None:
        if not ts or len(ts) != len(arrays):
            raise ValueError("n is required unless every array is a tensor")
        n = ts[0].numel()
        if any(t.numel() != n for t in ts):
            raise ValueError("shard tensors differ in length")
        return n
    n = int(n)
    for t in ts:
        if t.numel() < n:
            raise ValueError("n = %d exceeds a tensor of %d elements" % (n, t.numel()))
    return n


_raw_stream = None


def _stream(stream):
    """The hipStream_t of `stream` (a torch stream, a raw handle, or None for torch's current
    stream on the current device).  The current stream's handle is read without building a
    torch Stream object (which costs a few microseconds per call)."""
    global _raw_stream
    if stream is None:
        import torch
        if _raw_stream is None:
            getter = getattr(torch._C, "_cuda_getCurrentRawStream", None)
            _raw_stream = (lambda: getter(torch.cuda.current_device())) if getter is not None else \
                (lambda: torch.cuda.current_stream().cuda_stream)
        return _raw_stream()
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def zero_partition_layout(total_numel: int, nd: int, rank: int) -> Layout:
    out = Layout()
    _check(_lib.zero_partition_layout(total_numel, nd, rank, ctypes.byref(out)))
    return out


def zero_shard_step(grad16, master32, m32, v32, param16_out, lr, beta1, beta2, eps, weight_decay, step,
                    loss_scale, clip, n=None, stream=None) -> int:
    """Returns 0 (applied) or 1 (skipped on overflow); raises ZeroError on error.

    Arrays are torch device tensors (grad16/param16_out float16 or int16,
    master32/m32/v32 float32) or raw device addresses with an explicit n."""
    import torch
    h16 = (torch.float16, torch.int16)
    f32 = (torch.float32,)
    n = _shard_len(n, grad16, master32, m32, v32, param16_out)
    return _check(_lib.zero_shard_step(
        _addr(grad16, h16, "grad16"), _addr(master32, f32, "master32"), _addr(m32, f32, "m32"),
        _addr(v32, f32, "v32"), _addr(param16_out, h16, "param16_out"), int(n), float(lr), float(beta1),
        float(beta2), float(eps), float(weight_decay), int(step), float(loss_scale), float(clip),
        _stream(stream)))


class ShardStepCall:
    """zero_shard_step with its arrays, fixed hyperparameters and stream resolved once.

    For loops that step the same buffers many times (the gradient buffer refilled by the
    reduce-scatter, or one of a few such buffers): the tensors are checked here as
    zero_shard_step checks them, referenced for the object's lifetime (their storage must not
    be resized or swapped meanwhile), and each call passes only t, the loss scale and which
    gradient buffer to use (or, through `scaled`, a Scaler whose t and loss scale the library
    reads and updates).  The library still checks every array's allocation on every call.
    `stream` is taken now (None: torch's current stream at construction)."""

    def __init__(self, grads, master32, m32, v32, param16_out, lr, beta1, beta2, eps, weight_decay, clip,
                 stream=None):
        import torch
        h16, f32 = (torch.float16, torch.int16), (torch.float32,)
        grads = list(grads)
        if not grads:
            raise ValueError("at least one gradient buffer is needed")
        n = _shard_len(None, *grads, master32, m32, v32, param16_out)
        self._keep = (grads, master32, m32, v32, param16_out)
        self._grads = [ctypes.c_void_p(_addr(g, h16, "grad16")) for g in grads]
        self._rest = (ctypes.c_void_p(_addr(master32, f32, "master32")), ctypes.c_void_p(_addr(m32, f32, "m32")),
                      ctypes.c_void_p(_addr(v32, f32, "v32")), ctypes.c_void_p(_addr(param16_out, h16, "param16_out")),
                      ctypes.c_int64(n), _dbl(float(lr)), _dbl(float(beta1)), _dbl(float(beta2)), _dbl(float(eps)),
                      _dbl(float(weight_decay)))
        self._clip = _dbl(float(clip))
        self._stream = ctypes.c_void_p(_stream(stream))
        self._fn = _lib.zero_shard_step
        self.n = n
        # zero_step_args_t records, one per gradient buffer, for the scaler-driven call
        self._args = [StepArgs(g.value, *(a.value for a in self._rest), self._clip.value, self._stream.value)
                      for g in self._grads]
        self._args_addr = [ctypes.addressof(a) for a in self._args]
        self._scaled = _lib.zero_shard_step_scaled

    def __call__(self, step, loss_scale, which=0) -> int:
        """One step with t = step on gradient buffer `which`: 0 applied, 1 skipped."""
        rc = self._fn(self._grads[which], *self._rest, step, loss_scale, self._clip, self._stream)
        return _check(rc) if rc < 0 else rc

    def scaled(self, scaler, which=0) -> int:
        """One step on gradient buffer `which` at the scaler's t and loss scale, then the
        scaler's update, in one library call (zero_shard_step_scaled): 0 applied, 1 skipped."""
        rc = self._scaled(self._args_addr[which], scaler.addr)
        return _check(rc) if rc < 0 else rc


def zero_shard_step_noalloc(grad16, master32, m32, v32, param16_out, lr, beta1, beta2, eps, weight_decay, step,
                            loss_scale, clip, n=None, stream=None) -> int:
    """zero_shard_step through the allocation-free entry point (fixed per-GPU workspace;
    returns once the step has completed).  0 applied, 1 skipped; raises ZeroError."""
    import torch
    h16 = (torch.float16, torch.int16)
    f32 = (torch.float32,)
    n = _shard_len(n, grad16, master32, m32, v32, param16_out)
    return _check(_lib.zero_shard_step_noalloc(
        _addr(grad16, h16, "grad16"), _addr(master32, f32, "master32"), _addr(m32, f32, "m32"),
        _addr(v32, f32, "v32"), _addr(param16_out, h16, "param16_out"), int(n), float(lr), float(beta1),
        float(beta2), float(eps), float(weight_decay), int(step), float(loss_scale), float(clip),
        _stream(stream)))


def zero_shard_stats(grad16, n=None, stream=None) -> float:
    """Local sum of squares of a shard's loss-scaled fp16 gradients (fp64; inf/NaN on overflow)."""
    import torch
    n = _shard_len(n, grad16)
    out = ctypes.c_double()
    _check(_lib.zero_shard_stats(_addr(grad16, (torch.float16, torch.int16), "grad16"), int(n), ctypes.byref(out),
                                 _stream(stream)))
    return out.value


def zero_shard_apply(grad16, master32, m32, v32, param16_out, global_sumsq, lr, beta1, beta2, eps, weight_decay,
                     step, loss_scale, clip, n=None, stream=None) -> int:
    """The update with a caller-supplied global sum of squares; 0 applied, 1 skipped."""
    import torch
    h16 = (torch.float16, torch.int16)
    f32 = (torch.float32,)
    n = _shard_len(n, grad16, master32, m32, v32, param16_out)
    return _check(_lib.zero_shard_apply(
        _addr(grad16, h16, "grad16"), _addr(master32, f32, "master32"), _addr(m32, f32, "m32"),
        _addr(v32, f32, "v32"), _addr(param16_out, h16, "param16_out"), int(n), float(global_sumsq), float(lr),
        float(beta1), float(beta2), float(eps), float(weight_decay), int(step), float(loss_scale), float(clip),
        _stream(stream)))


def zero_shard_stats_async(grad16, local_sumsq, n=None, stream=None):
    """Enqueue the shard's sum of squares into local_sumsq (a float64 device tensor
    of one element, or a device address); returns without waiting."""
    import torch
    n = _shard_len(n, grad16)
    _check(_lib.zero_shard_stats_async(_addr(grad16, (torch.float16, torch.int16), "grad16"), int(n),
                                       _addr(local_sumsq, (torch.float64,), "local_sumsq"), _stream(stream)))


def zero_shard_apply_async(grad16, master32, m32, v32, param16_out, global_sumsq, lr, beta1, beta2, eps,
                           weight_decay, step, loss_scale, clip, skipped=None, n=None, stream=None):
    """Enqueue the update with the global sum read from device memory (global_sumsq:
    a float64 device tensor or address); the skip flag goes to `skipped` (an int32
    device tensor, a mapped host address, or None).  Returns without waiting."""
    import torch
    h16 = (torch.float16, torch.int16)
    f32 = (torch.float32,)
    n = _shard_len(n, grad16, master32, m32, v32, param16_out)
    _check(_lib.zero_shard_apply_async(
        _addr(grad16, h16, "grad16"), _addr(master32, f32, "master32"), _addr(m32, f32, "m32"),
        _addr(v32, f32, "v32"), _addr(param16_out, h16, "param16_out"), int(n),
        _addr(global_sumsq, (torch.float64,), "global_sumsq"), float(lr), float(beta1), float(beta2), float(eps),
        float(weight_decay), int(step), float(loss_scale), float(clip),
        _addr(skipped, (torch.int32,), "skipped"), _stream(stream)))


def resident_state_record(lr, beta1, beta2, eps, weight_decay, clip, loss_scale, min_scale=1.0, window=1000,
                          t=1) -> ResidentState:
    """A host zero_resident_state_t filled (and checked) by zero_resident_state_init."""
    st = ResidentState()
    _check(_lib.zero_resident_state_init(ctypes.addressof(st), float(lr), float(beta1), float(beta2), float(eps),
                                         float(weight_decay), float(clip), float(loss_scale), float(min_scale),
                                         int(window), int(t)))
    return st


def resident_state(device, lr, beta1, beta2, eps, weight_decay, clip, loss_scale, min_scale=1.0, window=1000, t=1):
    """A zero_resident_state_t record in device memory (a uint8 torch tensor), initialised
    from the host by zero_resident_state_init (which rejects out-of-range values)."""
    import torch
    st = resident_state_record(lr, beta1, beta2, eps, weight_decay, clip, loss_scale, min_scale, window, t)
    host = torch.frombuffer(bytearray(bytes(st)), dtype=torch.uint8)
    return host.to(device)


def zero_resident_release(state):
    """Free the resident step's workspace held for `state` (a device record tensor or address)."""
    _check(_lib.zero_resident_release(_addr(state, None, "state")))


def zero_stream_release(stream=None):
    """Free the library's workspace of `stream` (torch stream, raw handle, or None for the
    current stream) after its queued work."""
    _check(_lib.zero_stream_release(_stream(stream)))


def zero_workspace_count():
    """(per-stream workspaces, resident-record workspaces) the library holds."""
    a, b = _i64(), _i64()
    _check(_lib.zero_workspace_count(ctypes.byref(a), ctypes.byref(b)))
    return a.value, b.value


def read_resident_state(state_tensor) -> ResidentState:
    """The record's contents, copied to the host.  The copy is ordered after the work of
    torch's current stream only: after resident steps on another stream, synchronise that
    stream first."""
    return ResidentState.from_buffer_copy(bytes(state_tensor.cpu().numpy().tobytes()))


def zero_shard_step_resident(grad16, master32, m32, v32, param16_out, state, n=None, stream=None):
    """Enqueue one resident step (no host wait; capturable).  `state` is the device record
    from resident_state() or a raw device address."""
    import torch
    h16 = (torch.float16, torch.int16)
    f32 = (torch.float32,)
    n = _shard_len(n, grad16, master32, m32, v32, param16_out)
    if not isinstance(state, int) and state.numel() * state.element_size() < ctypes.sizeof(ResidentState):
        raise ValueError("state must hold a zero_resident_state_t (%d bytes)" % ctypes.sizeof(ResidentState))
    _check(_lib.zero_shard_step_resident(
        _addr(grad16, h16, "grad16"), _addr(master32, f32, "master32"), _addr(m32, f32, "m32"),
        _addr(v32, f32, "v32"), _addr(param16_out, h16, "param16_out"), int(n), _addr(state, None, "state"),
        _stream(stream)))


def zero_shard_validate(grad16, master32, m32, v32, param16_out, n):
    """zero_shard_step's array checks without launching anything; raises ZeroError."""
    return _check(_lib.zero_shard_validate(_addr(grad16), _addr(master32), _addr(m32), _addr(v32),
                                           _addr(param16_out), int(n)))


def zero_shard_last_stats():
    """(norm, mult, overflow) of the calling thread's last successful step."""
    norm, mult, ovf = _dbl(), ctypes.c_float(), ctypes.c_int()
    _check(_lib.zero_shard_last_stats(ctypes.byref(norm), ctypes.byref(mult), ctypes.byref(ovf)))
    return norm.value, mult.value, ovf.value


def zero_shard_last_step_stats() -> StepStats:
    """The whole statistics record of the calling thread's last successful step."""
    out = StepStats()
    _check(_lib.zero_shard_last_step_stats(ctypes.byref(out)))
    return out


def zero_bias_corrections(beta1, beta2, step):
    """The fp32 bias corrections (1 - beta1^t, 1 - beta2^t) the update kernels use (host only)."""
    a, b = ctypes.c_float(), ctypes.c_float()
    _check(_lib.zero_bias_corrections(float(beta1), float(beta2), int(step), ctypes.byref(a), ctypes.byref(b)))
    return a.value, b.value


class Scaler:
    """Dynamic loss scale kept in the library's zero_scaler_t."""

    def __init__(self, scale: float, window: int = 1000, min_scale: float = 1.0):
        self.state = ScalerState()
        _check(_lib.zero_scaler_init(ctypes.byref(self.state), scale, window, min_scale))
        self.addr = ctypes.addressof(self.state)  # for calls that update the scaler in the library

    @property
    def scale(self) -> float:
        return self.state.scale

    @property
    def t_next(self) -> int:
        return self.state.applied + 1

    def update(self, skipped):
        _check(_lib.zero_scaler_update(ctypes.byref(self.state), 1 if skipped else 0))


def zero_memory_bytes(psi: float, nd: int, stage: int, k: int = 12) -> float:
    out = ctypes.c_double()
    _check(_lib.zero_memory_bytes(float(psi), int(nd), int(stage), int(k), ctypes.byref(out)))
    return out.value


def zero_model_state_bytes(psi: float, nd: float, stage: int, k: float = 12.0) -> float:
    out = ctypes.c_double()
    _check(_lib.zero_model_state_bytes(psi, nd, stage, k, ctypes.byref(out)))
    return out.value


def zero_last_error() -> str:
    return _lib.zero_last_error().decode(errors="replace")


def zero_profile_enable(every):
    """Profile one step in `every` (True = every step, False/0 = off)."""
    _check(_lib.zero_profile_enable(int(every)))


def zero_profile_read() -> Profile:
    out = Profile()
    _check(_lib.zero_profile_read(ctypes.byref(out)))
    return out


def zero_probe_copy(src, dst, nbytes=None, stream=None):
    if nbytes is None:
        nbytes = src.numel() * src.element_size()
    for t in (src, dst):
        if not isinstance(t, int) and t.numel() * t.element_size() < nbytes:
            raise ValueError("nbytes = %d exceeds a buffer of %d bytes" % (nbytes, t.numel() * t.element_size()))
    _check(_lib.zero_probe_copy(_addr(src), _addr(dst), int(nbytes), _stream(stream)))


def zero_probe_adam_mix(grad16, master32, m32, v32, param16_out, n=None, stream=None):
    """Enqueue the byte-mix probe of the Adam update over the arrays (it overwrites master32,
    m32, v32 and param16_out)."""
    import torch
    h16 = (torch.float16, torch.int16)
    f32 = (torch.float32,)
    n = _shard_len(n, grad16, master32, m32, v32, param16_out)
    _check(_lib.zero_probe_adam_mix(_addr(grad16, h16, "grad16"), _addr(master32, f32, "master32"),
                                    _addr(m32, f32, "m32"), _addr(v32, f32, "v32"),
                                    _addr(param16_out, h16, "param16_out"), int(n), _stream(stream)))


def zero_probe_lamb_pass(pass_, grad16, master32, m32, v32, param16_out, n=None, stream=None):
    """Enqueue the byte-mix probe of LAMB pass `pass_` (0 moments, 1 apply) over the arrays
    (it overwrites what that pass writes)."""
    n = _shard_len(n, *(a for a in (grad16, master32, m32, v32, param16_out) if a is not None))
    _check(_lib.zero_probe_lamb_pass(int(pass_), _addr(grad16), _addr(master32), _addr(m32), _addr(v32),
                                     _addr(param16_out), int(n), _stream(stream)))


class LambPlan:
    """A LAMB layer-table plan (zero_lamb_plan_t) on the current device.

    seg_off: the n_seg + 1 layer offsets of the shard (any int sequence or
    int64 array, copied by the library); n = seg_off[-1]."""

    def __init__(self, seg_off):
        import numpy as np
        off = np.ascontiguousarray(np.asarray(seg_off, dtype=np.int64))
        if off.ndim != 1 or off.size < 1:
            raise ValueError("seg_off must be a 1-D sequence of n_seg + 1 offsets")
        self.n = int(off[-1])
        self.n_seg = off.size - 1
        h = _P()
        _check(_lib.zero_lamb_plan_create(off.ctypes.data, self.n_seg, self.n, ctypes.byref(h)))
        self._h = h

    @property
    def handle(self):
        return self._h

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            h, self._h = self._h, None
            _check(_lib.zero_lamb_plan_destroy(h))

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _lamb_check_len(plan, *tensors):
    for t in tensors:
        if t is not None and not isinstance(t, int) and t.numel() != plan.n:
            raise ValueError("shard tensors must have the plan's n = %d elements" % plan.n)


def zero_lamb_step(plan, grad16, master32, m32, v32, param16_out, lr, beta1, beta2, eps, weight_decay, step,
                   loss_scale, clip, phi_lo=0.0, phi_hi=float("inf"), stream=None) -> int:
    """One LAMB step over the plan's layers; 0 applied, 1 skipped (overflow)."""
    import torch
    h16, f32 = (torch.float16, torch.int16), (torch.float32,)
    _lamb_check_len(plan, grad16, master32, m32, v32, param16_out)
    return _check(_lib.zero_lamb_step(
        plan.handle, _addr(grad16, h16, "grad16"), _addr(master32, f32, "master32"), _addr(m32, f32, "m32"),
        _addr(v32, f32, "v32"), _addr(param16_out, h16, "param16_out"), float(lr), float(beta1), float(beta2),
        float(eps), float(weight_decay), int(step), float(loss_scale), float(clip), float(phi_lo), float(phi_hi),
        _stream(stream)))


def zero_lamb_moments(plan, grad16, master32, m32, v32, global_sumsq, beta1, beta2, eps, weight_decay, step,
                      loss_scale, clip, layer_sumsq, stream=None) -> int:
    """Split phase, part 1: moments and this shard's per-layer sums into
    layer_sumsq (a float64 device tensor of 2*n_seg elements)."""
    import torch
    h16, f32 = (torch.float16, torch.int16), (torch.float32,)
    _lamb_check_len(plan, grad16, master32, m32, v32)
    if not isinstance(layer_sumsq, int) and layer_sumsq.numel() != 2 * plan.n_seg:
        raise ValueError("layer_sumsq must hold 2 * n_seg = %d doubles" % (2 * plan.n_seg))
    return _check(_lib.zero_lamb_moments(
        plan.handle, _addr(grad16, h16, "grad16"), _addr(master32, f32, "master32"), _addr(m32, f32, "m32"),
        _addr(v32, f32, "v32"), float(global_sumsq), float(beta1), float(beta2), float(eps), float(weight_decay),
        int(step), float(loss_scale), float(clip), _addr(layer_sumsq, (torch.float64,), "layer_sumsq"),
        _stream(stream)))


def zero_lamb_apply(plan, master32, m32, v32, param16_out, global_sumsq, layer_sumsq, lr, beta1, beta2, eps,
                    weight_decay, step, phi_lo=0.0, phi_hi=float("inf"), stream=None) -> int:
    """Split phase, part 2: the update from the stored moments and the completed layer sums."""
    import torch
    h16, f32 = (torch.float16, torch.int16), (torch.float32,)
    _lamb_check_len(plan, master32, m32, v32, param16_out)
    if not isinstance(layer_sumsq, int) and layer_sumsq.numel() != 2 * plan.n_seg:
        raise ValueError("layer_sumsq must hold 2 * n_seg = %d doubles" % (2 * plan.n_seg))
    return _check(_lib.zero_lamb_apply(
        plan.handle, _addr(master32, f32, "master32"), _addr(m32, f32, "m32"), _addr(v32, f32, "v32"),
        _addr(param16_out, h16, "param16_out"), float(global_sumsq), _addr(layer_sumsq, (torch.float64,),
                                                                           "layer_sumsq"),
        float(lr), float(beta1), float(beta2), float(eps), float(weight_decay), int(step), float(phi_lo),
        float(phi_hi), _stream(stream)))


def zero_lamb_profile_read() -> LambProfile:
    out = LambProfile()
    _check(_lib.zero_lamb_profile_read(ctypes.byref(out)))
    return out


def raw_library():
    """The loaded ctypes library (for ABI-level tests)."""
    return _lib
