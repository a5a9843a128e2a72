"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Bit-exact: layout, the skip flag, the loss-scale sequence and t.  Floating
point after every step: master, m and v within max|d| <= 1e-6 * max(1, |x|) of
the oracle, fp16 parameters within 1 ulp (sign-magnitude order).  Guard
canaries around every device buffer must stay intact.  Bitwise agreement of
the floating-point state is recorded as a diagnostic.
"""
import json
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import gpu_harness as H  # noqa: E402

import oracle  # noqa: E402
from paper_1910_02054_amd import workloads  # noqa: E402

pytestmark = pytest.mark.gpu


def say(*a):
    print("[gpu-parity]", *a, flush=True)


@pytest.fixture(scope="module")
def env():
    import torch
    from paper_1910_02054_amd import binding
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch, binding, torch.device("cuda:0")


def _alloc(torch, dev, n, shifts=(0, 0, 0, 0, 0)):
    return [H.Guarded(torch, n, torch.float16, dev, shifts[0]), H.Guarded(torch, n, torch.float32, dev, shifts[1]),
            H.Guarded(torch, n, torch.float32, dev, shifts[2]), H.Guarded(torch, n, torch.float32, dev, shifts[3]),
            H.Guarded(torch, n, torch.float16, dev, shifts[4])]


def _run_case(env, g16_steps, theta, m, v, hp, scales=None, shifts=(0, 0, 0, 0, 0), clip=1.0, t0=1, label=""):
    """Run a sequence of steps on the GPU and in the oracle from the same inputs."""
    torch, zb, dev = env
    n = theta.size
    bufs = _alloc(torch, dev, n, shifts)
    bufs[1].upload(theta)
    bufs[2].upload(m)
    bufs[3].upload(v)
    bufs[4].upload(workloads.p16_sentinel(n))
    ref = [theta.copy(), m.copy(), v.copy(), workloads.p16_sentinel(n)]
    diags = []
    for k, g16 in enumerate(g16_steps):
        scale = scales[k] if scales else 2.0 ** 16
        t = t0 + k
        bufs[0].upload(g16)
        say(label, "step", k + 1, "n", n, "shifts", shifts)
        flag = zb.zero_shard_step(bufs[0].view, bufs[1].view, bufs[2].view, bufs[3].view, bufs[4].view,
                                  hp["lr"], hp["beta1"], hp["beta2"], hp["eps"], hp["wd"], t, scale, clip)
        st = zb.zero_shard_last_step_stats()
        torch.cuda.synchronize()
        skip, sc = H.oracle_step(g16, *ref, hp["lr"], hp["beta1"], hp["beta2"], hp["eps"], hp["wd"], t, scale, clip)
        assert flag == skip and st.skipped == skip and st.overflow == skip
        gpu = [b.download() for b in bufs[1:]]
        d = H.compare_state(gpu, ref)
        if not skip:
            d["norm_rel"] = abs(st.norm / sc.norm - 1.0) if sc.norm > 0 else abs(st.norm)
            d["mult_equal"] = bool(np.float32(st.mult) == np.float32(sc.mult))
            assert d["norm_rel"] <= 1e-9
        assert all(b.guards_intact() for b in bufs), "guard canaries overwritten"
        diags.append(d)
    return diags, ref


HP_W = lambda w: dict(lr=w.lr, beta1=w.beta1, beta2=w.beta2, eps=w.eps, wd=w.weight_decay)  # noqa: E731


def _run_workload(env, key, steps=None, rank=None):
    torch, zb, dev = env
    w = workloads.WORKLOADS[key]
    r = w.rank if rank is None else rank
    lay = zb.zero_partition_layout(w.psi, w.nd, r)
    assert (lay.shard_numel, lay.offset, lay.valid_numel, lay.padded_total) == oracle.layout(w.psi, w.nd, r)
    n = lay.valid_numel
    theta, m, v = workloads.initial_state(w, n)
    nsteps = steps or w.steps
    # the shard keeps the alignment it has inside a flat buffer: offset mod 8 elements
    shift = lay.offset % 8
    bufs = _alloc(torch, dev, n, (shift,) * 5)
    say(key, "n", n, "offset mod 8", shift, "steps", nsteps)
    for b, a in zip(bufs[1:4], (theta, m, v)):
        b.upload(a)
    bufs[4].upload(workloads.p16_sentinel(n))
    ref = [theta, m, v, workloads.p16_sentinel(n)]
    s_gpu, s_ora = zb.Scaler(w.loss_scale), oracle.Scaler(w.loss_scale)
    hp = HP_W(w)
    log = []
    for step in range(1, nsteps + 1):
        assert s_gpu.scale == s_ora.scale.value and s_gpu.t_next == s_ora.t_next
        scale, t = s_gpu.scale, s_gpu.t_next
        g16 = workloads.gradients(w, n, step, scale)
        bufs[0].upload(g16)
        say(key, "step", step, "t", t, "scale", scale)
        flag = zb.zero_shard_step(bufs[0].view, bufs[1].view, bufs[2].view, bufs[3].view, bufs[4].view,
                                  hp["lr"], hp["beta1"], hp["beta2"], hp["eps"], hp["wd"], t, scale, w.clip)
        st = zb.zero_shard_last_step_stats()
        torch.cuda.synchronize()
        skip, sc = H.oracle_step(g16, *ref, hp["lr"], hp["beta1"], hp["beta2"], hp["eps"], hp["wd"], t, scale, w.clip)
        assert flag == skip, (step, flag, skip)
        s_gpu.update(flag)
        s_ora.update(skip)
        gpu = [b.download() for b in bufs[1:]]
        d = H.compare_state(gpu, ref)
        d.update(step=step, skip=int(flag), t=t, scale=scale)
        if not skip:
            d["norm_rel"] = abs(st.norm / sc.norm - 1.0)
            d["mult_equal"] = bool(np.float32(st.mult) == np.float32(sc.mult))
            d["coef"] = sc.coef
            assert d["norm_rel"] <= 1e-9
        assert all(b.guards_intact() for b in bufs)
        log.append(d)
        say(json.dumps(d))
    return log, s_gpu


def test_tiny_workload(env):
    log, sc = _run_workload(env, "tiny")
    assert [d["skip"] for d in log] == [0, 0, 0]
    assert all(d["coef"] < 1.0 for d in log)  # clipping active


@pytest.mark.parametrize("key", ["gpt2_1p5b", "dp_13b", "mp16_dp25_100b"])
def test_large_workloads(env, key):
    log, sc = _run_workload(env, key)
    assert not any(d["skip"] for d in log)
    assert sc.state.applied == workloads.WORKLOADS[key].steps


def test_ragged_overflow_workload(env):
    log, sc = _run_workload(env, "ragged_1t")
    assert [d["step"] for d in log if d["skip"]] == [3, 7]
    assert sc.scale == 2.0 ** 14 and sc.state.applied == 10


def test_ragged_workload_rank0_full_shard(env):
    log, _ = _run_workload(env, "ragged_1t", steps=4, rank=0)
    assert [d["skip"] for d in log] == [0, 0, 1, 0]


EDGE_NS = [1, 2, 3, 4, 5, 7, 8, 9, 15, 16, 17, 31, 33, 255, 256, 257, 1023, 1024, 1025, 2047, 2048, 2049,
           8 * 256 * 4 - 1, 8 * 256 * 4 + 3, 100_003, 1_000_003]


@pytest.mark.parametrize("n", EDGE_NS)
def test_sizes_and_tails(env, n):
    g16, theta, m, v = workloads.random_case(1000 + n, n)
    hp = dict(lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.0)
    _run_case(env, [g16, g16[::-1].copy()], theta, m, v, hp, label="n=%d" % n)


@pytest.mark.parametrize("shifts", [(1, 1, 1, 1, 1), (2, 2, 2, 2, 2), (3, 3, 3, 3, 3), (5, 5, 5, 5, 5),
                                    (7, 7, 7, 7, 7), (0, 1, 0, 0, 0), (1, 0, 2, 3, 0), (0, 0, 0, 0, 3)])
def test_misaligned_views(env, shifts):
    n = 50_001
    g16, theta, m, v = workloads.random_case(77, n)
    hp = dict(lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.0)
    _run_case(env, [g16], theta, m, v, hp, shifts=shifts, label="shifts")


@pytest.mark.parametrize("case", ["wd", "noclip", "beta0", "lr0", "scale_odd", "late_t", "subnormal_out"])
def test_hyperparameter_cases(env, case):
    n = 70_001
    g16, theta, m, v = workloads.random_case(88, n, loss_scale=1000.0 if case == "scale_odd" else 2.0 ** 16)
    hp = dict(lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.0)
    clip, t0, scales = 1.0, 1, [2.0 ** 16] * 2
    if case == "wd":
        hp["wd"] = 0.01
    elif case == "noclip":
        clip = 0.0
    elif case == "beta0":
        hp.update(beta1=0.0, beta2=0.0)
    elif case == "lr0":
        hp["lr"] = 0.0
    elif case == "scale_odd":
        scales = [1000.0, 1000.0]
    elif case == "late_t":
        t0 = 12345
    elif case == "subnormal_out":
        theta[:] = np.float32(3e-6) * (np.arange(n, dtype=np.float32) % 50 - 25)
    _run_case(env, [g16, g16], theta, m, v, hp, scales=scales, clip=clip, t0=t0, label=case)


@pytest.mark.parametrize("where,pattern", [("last", 0x7C00), ("first", 0x7E01), ("middle", 0xFC00),
                                           ("first", 0xFFFF), ("last", 0x7D00)])
def test_overflow_skips_and_touches_nothing(env, where, pattern):
    torch, zb, dev = env
    n = 33_333
    g16, theta, m, v = workloads.random_case(99, n)
    pos = {"first": 0, "last": n - 1, "middle": n // 2}[where]
    g16[pos] = pattern
    bufs = _alloc(torch, dev, n)
    for b, a in zip(bufs, (g16, theta, m, v, workloads.p16_sentinel(n))):
        b.upload(a)
    say("overflow", where, hex(pattern))
    flag = zb.zero_shard_step(bufs[0].view, bufs[1].view, bufs[2].view, bufs[3].view, bufs[4].view,
                              1e-4, 0.9, 0.999, 1e-8, 0.0, 1, 2.0 ** 16, 1.0)
    torch.cuda.synchronize()
    assert flag == 1
    st = zb.zero_shard_last_step_stats()
    assert st.overflow == 1 and st.skipped == 1
    for b, a in zip(bufs[1:], (theta, m, v, workloads.p16_sentinel(n))):
        got = b.download()
        assert np.array_equal(got.view(np.uint8), np.ascontiguousarray(a).view(np.uint8))
    assert all(b.guards_intact() for b in bufs)


def test_deterministic_run_to_run(env):
    torch, zb, dev = env
    n = 2_000_003
    g16, theta, m, v = workloads.random_case(5, n)
    outs = []
    for rep in range(2):
        bufs = _alloc(torch, dev, n)
        for b, a in zip(bufs, (g16, theta, m, v, workloads.p16_sentinel(n))):
            b.upload(a)
        say("determinism rep", rep)
        zb.zero_shard_step(bufs[0].view, bufs[1].view, bufs[2].view, bufs[3].view, bufs[4].view,
                           1e-4, 0.9, 0.999, 1e-8, 0.0, 1, 2.0 ** 16, 1.0)
        st = zb.zero_shard_last_step_stats()
        torch.cuda.synchronize()
        outs.append(([b.download().copy() for b in bufs[1:]], st.sumsq, st.mult))
    for a, b in zip(outs[0][0], outs[1][0]):
        assert np.array_equal(a.view(np.uint8), b.view(np.uint8))
    assert outs[0][1] == outs[1][1] and outs[0][2] == outs[1][2]


def test_zero_elements_touches_nothing(env):
    torch, zb, dev = env
    bufs = _alloc(torch, dev, 0)
    flag = zb.zero_shard_step(bufs[0].view, bufs[1].view, bufs[2].view, bufs[3].view, bufs[4].view,
                              1e-4, 0.9, 0.999, 1e-8, 0.0, 1, 2.0 ** 16, 1.0)
    torch.cuda.synchronize()
    assert flag == 0 and all(b.guards_intact() for b in bufs)


def test_side_stream(env):
    torch, zb, dev = env
    n = 300_007
    g16, theta, m, v = workloads.random_case(6, n)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        bufs = _alloc(torch, dev, n)
        for b, a in zip(bufs, (g16, theta, m, v, workloads.p16_sentinel(n))):
            b.upload(a)
        say("side stream")
        flag = zb.zero_shard_step(bufs[0].view, bufs[1].view, bufs[2].view, bufs[3].view, bufs[4].view,
                                  1e-4, 0.9, 0.999, 1e-8, 0.0, 1, 2.0 ** 16, 1.0, stream=s)
    s.synchronize()
    ref = [theta.copy(), m.copy(), v.copy(), workloads.p16_sentinel(n)]
    skip, _ = H.oracle_step(g16, *ref, 1e-4, 0.9, 0.999, 1e-8, 0.0, 1, 2.0 ** 16, 1.0)
    assert flag == skip == 0
    H.compare_state([b.download() for b in bufs[1:]], ref)


def test_probe_copy(env):
    torch, zb, dev = env
    src = torch.randint(0, 1 << 30, (1 << 20,), dtype=torch.int32, device=dev)
    dst = torch.zeros_like(src)
    zb.zero_probe_copy(src, dst)
    torch.cuda.synchronize()
    assert torch.equal(src, dst)


def test_profile_counts_steps(env):
    torch, zb, dev = env
    n = 1 << 20
    g16, theta, m, v = workloads.random_case(7, n)
    bufs = _alloc(torch, dev, n)
    for b, a in zip(bufs, (g16, theta, m, v, workloads.p16_sentinel(n))):
        b.upload(a)
    zb.zero_profile_read()
    zb.zero_profile_enable(True)
    for t in range(1, 4):
        zb.zero_shard_step(bufs[0].view, bufs[1].view, bufs[2].view, bufs[3].view, bufs[4].view,
                           1e-4, 0.9, 0.999, 1e-8, 0.0, t, 2.0 ** 16, 1.0)
    zb.zero_profile_enable(False)
    p = zb.zero_profile_read()
    assert p.steps == 3 and p.stats_ms > 0 and p.update_ms > 0


def test_profile_samples_one_step_in_k(env):
    torch, zb, dev = env
    n = 1 << 20
    g16, theta, m, v = workloads.random_case(8, n)
    bufs = _alloc(torch, dev, n)
    for b, a in zip(bufs, (g16, theta, m, v, workloads.p16_sentinel(n))):
        b.upload(a)
    zb.zero_profile_read()
    zb.zero_profile_enable(3)
    for t in range(1, 8):
        zb.zero_shard_step(bufs[0].view, bufs[1].view, bufs[2].view, bufs[3].view, bufs[4].view,
                           1e-4, 0.9, 0.999, 1e-8, 0.0, t, 2.0 ** 16, 1.0)
    zb.zero_profile_enable(0)
    p = zb.zero_profile_read()
    assert p.steps == 3 and p.update_ms > 0  # steps 1, 4 and 7


def test_checkpoint_resume_equals_straight_run(env, tmp_path):
    # The state is exactly master/m/v (+ the scaler's t and scale): saving it after 5 steps
    # and resuming in fresh buffers gives the same bytes as 10 uninterrupted steps.
    torch, zb, dev = env
    n = 500_003
    grads = [workloads.random_case(300 + k, n)[0] for k in range(10)]
    _, theta, m, v = workloads.random_case(299, n)

    def run(state, ks, t0):
        bufs = _alloc(torch, dev, n)
        for b, a in zip(bufs[1:4], state):
            b.upload(a)
        bufs[4].upload(workloads.p16_sentinel(n))
        for k in ks:
            bufs[0].upload(grads[k])
            assert zb.zero_shard_step(*(b.view for b in bufs), 1e-4, 0.9, 0.999, 1e-8, 0.0, t0 + k, 2.0 ** 16,
                                      1.0) == 0
        torch.cuda.synchronize()
        return [b.download().copy() for b in bufs[1:]]

    straight = run((theta, m, v), range(10), 1)
    first = run((theta, m, v), range(5), 1)
    np.savez(tmp_path / "ckpt.npz", master=first[0], m=first[1], v=first[2])
    ck = np.load(tmp_path / "ckpt.npz")
    resumed = run((ck["master"], ck["m"], ck["v"]), range(5, 10), 1)
    for a, b in zip(straight, resumed):
        assert np.array_equal(a.view(np.uint8), b.view(np.uint8))


@pytest.mark.parametrize("same_stream", [False, True])
def test_concurrent_host_threads(env, same_stream):
    # Calls overlap in the library (ctypes releases the GIL): each stream has its own workspace,
    # and calls that share a stream are serialised.  Every thread's result must match the oracle.
    import threading
    torch, zb, dev = env
    n = 400_009
    shared = torch.cuda.Stream()
    cases = []
    for k in range(3):
        g16, theta, m, v = workloads.random_case(400 + k, n)
        bufs = _alloc(torch, dev, n)
        for b, a in zip(bufs, (g16, theta, m, v, workloads.p16_sentinel(n))):
            b.upload(a)
        cases.append((bufs, [theta.copy(), m.copy(), v.copy(), workloads.p16_sentinel(n)], g16))
    torch.cuda.synchronize()
    errors = []

    def work(k):
        try:
            bufs, _, _ = cases[k]
            s = shared if same_stream else torch.cuda.Stream()
            for t in range(1, 4):
                f = zb.zero_shard_step(*(b.view for b in bufs), 1e-4, 0.9, 0.999, 1e-8, 0.0, t, 2.0 ** 16, 1.0,
                                       stream=s)
                assert f == 0
            s.synchronize()
        except Exception as e:  # reported below
            errors.append(e)

    threads = [threading.Thread(target=work, args=(k,)) for k in range(3)]
    say("concurrent threads, same stream:", same_stream)
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for bufs, ref, g16 in cases:
        for t in range(1, 4):
            H.oracle_step(g16, *ref, 1e-4, 0.9, 0.999, 1e-8, 0.0, t, 2.0 ** 16, 1.0)
        H.compare_state([b.download() for b in bufs[1:]], ref)
        assert all(b.guards_intact() for b in bufs)


def test_validate_catches_overruns_and_host_memory(env):
    # Only zero_shard_validate is called with bad arguments: nothing is ever launched on them.
    torch, zb, dev = env
    n = 1000
    bufs = _alloc(torch, dev, n)
    views = [b.view for b in bufs]
    assert zb.zero_shard_validate(*views, n) == 0
    with pytest.raises(zb.ZeroError) as e:
        zb.zero_shard_validate(*views, 10 ** 9)
    assert e.value.code == zb.ZERO_EINVAL and "overruns" in str(e.value)
    host = [np.zeros(n, np.uint16), np.zeros(n, np.float32), np.zeros(n, np.float32), np.zeros(n, np.float32),
            np.zeros(n, np.uint16)]
    with pytest.raises(zb.ZeroError) as e:
        zb.zero_shard_validate(*(h.ctypes.data for h in host), n)
    assert e.value.code == zb.ZERO_EINVAL


def test_reallocated_smaller_buffer_is_rejected(env):
    # The allocation check runs on every call: after a step on five 8M-element buffers, the
    # gradient buffer is freed and a 1 MiB one allocated (often at the same address); a step
    # with the old n must be refused before any launch.  Raw hipMalloc/hipFree, outside torch's
    # caching allocator, so the allocations are exactly the requested sizes.
    import ctypes
    torch, zb, dev = env
    # the HIP runtime already in the process (torch and the library share it): never a second copy
    hip = ctypes.CDLL("libamdhip64.so.7", mode=os.RTLD_NOLOAD)
    hip.hipMalloc.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_size_t]
    hip.hipFree.argtypes = [ctypes.c_void_p]
    hip.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
    n = 8 << 20
    sizes = (2 * n, 4 * n, 4 * n, 4 * n, 2 * n)
    ptrs = []
    for sz in sizes:
        p = ctypes.c_void_p()
        assert hip.hipMalloc(ctypes.byref(p), sz) == 0
        ptrs.append(p.value)
    try:
        zero16 = torch.zeros(n, dtype=torch.float16, device=dev)
        zero32 = torch.zeros(n, dtype=torch.float32, device=dev)
        for i, p in enumerate(ptrs):  # defined contents: zero gradients and state
            src = zero16 if sizes[i] == 2 * n else zero32
            assert hip.hipMemcpy(p, src.data_ptr(), sizes[i], 3) == 0  # device to device
        torch.cuda.synchronize()
        assert zb.zero_shard_step(*ptrs, 1e-4, 0.9, 0.999, 1e-8, 0.0, 1, 1.0, 0.0, n=n) == 0
        torch.cuda.synchronize()
        old = ptrs[0]
        assert hip.hipFree(ptrs[0]) == 0
        p = ctypes.c_void_p()
        assert hip.hipMalloc(ctypes.byref(p), 1 << 20) == 0
        ptrs[0] = p.value
        say("re-allocated gradient buffer", "at the same address" if p.value == old else "elsewhere")
        with pytest.raises(zb.ZeroError) as e:
            zb.zero_shard_step(*ptrs, 1e-4, 0.9, 0.999, 1e-8, 0.0, 2, 1.0, 0.0, n=n)
        assert e.value.code == zb.ZERO_EINVAL and "overruns" in str(e.value)
        with pytest.raises(zb.ZeroError):
            zb.zero_shard_apply(*ptrs, 0.0, 1e-4, 0.9, 0.999, 1e-8, 0.0, 2, 1.0, 0.0, n=n)
    finally:
        torch.cuda.synchronize()
        for p in ptrs:
            hip.hipFree(p)


def test_workspace_does_not_grow_with_the_shard(env):
    # Sec. 6.2's constant-size buffers: the library's own device memory for a step is a
    # fixed-size workspace per (device, stream), whatever n is.  Device free memory is read
    # through the HIP runtime around single calls on fresh streams (first a 1M-element shard,
    # then a 200M-element one); no Psi-sized temporary may appear.
    import ctypes
    torch, zb, dev = env
    hip = ctypes.CDLL("libamdhip64.so.7", mode=os.RTLD_NOLOAD)
    hip.hipMemGetInfo.argtypes = [ctypes.POINTER(ctypes.c_size_t), ctypes.POINTER(ctypes.c_size_t)]

    def free_bytes():
        torch.cuda.synchronize()
        f, t = ctypes.c_size_t(), ctypes.c_size_t()
        assert hip.hipMemGetInfo(ctypes.byref(f), ctypes.byref(t)) == 0
        return f.value

    deltas = {}
    for n in (1 << 20, 200_000_000):
        bufs = _alloc(torch, dev, n)
        for b, a in zip(bufs, (np.zeros(n, np.uint16), np.zeros(n, np.float32), np.zeros(n, np.float32),
                               np.zeros(n, np.float32), np.zeros(n, np.uint16))):
            b.upload(a)
        s = torch.cuda.Stream()
        before = free_bytes()
        flag = zb.zero_shard_step(*(b.view for b in bufs), 1e-4, 0.9, 0.999, 1e-8, 0.0, 1, 1.0, 0.0, stream=s)
        s.synchronize()
        deltas[n] = before - free_bytes()
        say("workspace on a fresh stream, n", n, "device bytes", deltas[n])
        assert flag == 0
        del bufs
        torch.cuda.empty_cache()
    # nothing proportional to n: one byte per element would already be 200 MB at the larger size
    assert all(d < (16 << 20) for d in deltas.values()), deltas


def test_loss_scale_too_large_overflows_then_recovers(env):
    # Dynamic loss scaling's own failure mode: at 2^24 the fp16 cast of the scaled gradients
    # overflows (inf in the generated gradient itself, not an injected one), so the step skips
    # and the scaler halves the scale, and keeps halving while the gradients still overflow;
    # the first scale at which they fit applies the step, which must match the oracle.
    torch, zb, dev = env
    n = 200_003
    _, theta, m, v = workloads.random_case(77, n)
    bufs = _alloc(torch, dev, n)
    for b, a in zip(bufs[1:], (theta, m, v, workloads.p16_sentinel(n))):
        b.upload(a)
    ref = [theta.copy(), m.copy(), v.copy(), workloads.p16_sentinel(n)]
    scaler = zb.Scaler(2.0 ** 24)
    flags = []
    for _ in range(12):
        scale = scaler.scale
        g16 = workloads.random_case(78, n, grad_std=0.05, loss_scale=scale)[0]   # same gradient, rescaled
        bufs[0].upload(g16)
        flag = zb.zero_shard_step(*(b.view for b in bufs), 1e-4, 0.9, 0.999, 1e-8, 0.0, scaler.t_next, scale, 1.0)
        torch.cuda.synchronize()
        skip, _ = H.oracle_step(g16, *ref, 1e-4, 0.9, 0.999, 1e-8, 0.0, scaler.t_next, scale, 1.0)
        assert flag == skip
        flags.append(flag)
        scaler.update(flag)
        H.compare_state([b.download() for b in bufs[1:]], ref)
        if not flag:
            break
    say("scale sequence flags", flags, "applied at scale", scale)
    assert flags[0] == 1 and flags[-1] == 0 and scaler.t_next == 2
    assert all(b.guards_intact() for b in bufs)


def test_step_waits_behind_queued_work(env):
    # Work queued ahead of the step on its stream (a bounded spin kernel of about 50 ms) makes the
    # host wait long enough to leave the spinning phase and poll with sleeps; the step's result
    # is unchanged.
    import time
    torch, zb, dev = env
    n = 100_003
    g16, theta, m, v = workloads.random_case(61, n)
    bufs = _alloc(torch, dev, n)
    for b, a in zip(bufs, (g16, theta, m, v, workloads.p16_sentinel(n))):
        b.upload(a)
    ref = [theta.copy(), m.copy(), v.copy(), workloads.p16_sentinel(n)]
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        torch.cuda._sleep(120_000_000)   # clock cycles
        t0 = time.perf_counter()
        flag = zb.zero_shard_step(*(b.view for b in bufs), 1e-4, 0.9, 0.999, 1e-8, 0.0, 1, 2.0 ** 16, 1.0)
        waited = time.perf_counter() - t0
    s.synchronize()
    say("host wait behind queued work: %.1f ms" % (waited * 1e3))
    skip, _ = H.oracle_step(g16, *ref, 1e-4, 0.9, 0.999, 1e-8, 0.0, 1, 2.0 ** 16, 1.0)
    assert flag == skip == 0
    H.compare_state([b.download() for b in bufs[1:]], ref)
    assert all(b.guards_intact() for b in bufs)
