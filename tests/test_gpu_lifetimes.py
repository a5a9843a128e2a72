"""GPU tests of the library's workspaces and of cross-stream ordering.

* Per-stream workspaces have a lifetime: 1,000 streams each take a step and
  are released; the library's count returns to where it started and device
  free memory comes back.
* The resident step's workspace belongs to its state record: two graphs
  captured on one stream with two records are replayed at the same time on
  two other streams, while eager steps run on the capture stream, and every
  result equals the eager resident steps of the same records.
* A LAMB plan moved between two streams orders itself with its own event:
  while a third stream is busy for about 50 ms, calls that alternate between
  the two streams return without waiting for it, and every step matches the
  oracle.
* A resident record whose hyperparameters are out of range is not a step:
  nothing is written and its skipped field reads -1.
* The LAMB byte-mix probes touch exactly their arrays' [0, n) and compute
  what they state.
"""
import ctypes
import os
import sys
import time

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import gpu_harness as H  # noqa: E402

import oracle  # noqa: E402
from paper_1910_02054_amd import workloads  # noqa: E402

pytestmark = pytest.mark.gpu
HP = dict(lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0, clip=1.0)


def say(*a):
    print("[gpu-lifetimes]", *a, flush=True)


@pytest.fixture(scope="module")
def env():
    import torch
    from paper_1910_02054_amd import binding
    assert torch.cuda.is_available()
    return torch, binding, torch.device("cuda:0")


def _alloc(torch, dev, n):
    dts = (torch.float16, torch.float32, torch.float32, torch.float32, torch.float16)
    return [H.Guarded(torch, n, dt, dev) for dt in dts]


def _hip():
    import torch
    path = None
    for cand in ("libamdhip64.so", os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "lib", "libamdhip64.so")):
        try:
            lib = ctypes.CDLL(cand)
            path = cand
            break
        except OSError:
            continue
    assert path is not None, "libamdhip64.so not found"
    lib.hipStreamCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
    lib.hipStreamDestroy.argtypes = [ctypes.c_void_p]
    lib.hipStreamSynchronize.argtypes = [ctypes.c_void_p]
    del torch
    return lib


def test_stream_workspaces_are_released(env):
    torch, zb, dev = env
    hip = _hip()
    n = 4099
    g16, theta, m, v = workloads.random_case(5000, n)
    bufs = _alloc(torch, dev, n)
    for b, a in zip(bufs, (g16, theta, m, v, workloads.p16_sentinel(n))):
        b.upload(a)
    torch.cuda.synchronize()
    streams0, _ = zb.zero_workspace_count()
    free0 = torch.cuda.mem_get_info()[0]
    handles = []
    for k in range(1000):
        h = ctypes.c_void_p()
        assert hip.hipStreamCreate(ctypes.byref(h)) == 0
        handles.append(h.value)
        assert zb.zero_shard_step(*(b.view for b in bufs), 1e-6, 0.9, 0.999, 1e-8, 0.0, 1, 2.0 ** 16, 1.0,
                                  stream=h.value) == 0
    grown, _ = zb.zero_workspace_count()
    free_mid = torch.cuda.mem_get_info()[0]
    say("workspaces", streams0, "->", grown, "free MiB", free0 >> 20, "->", free_mid >> 20)
    assert grown == streams0 + 1000
    for h in handles:
        zb.zero_stream_release(h)
        assert hip.hipStreamDestroy(ctypes.c_void_p(h)) == 0
    after, _ = zb.zero_workspace_count()
    free1 = torch.cuda.mem_get_info()[0]
    say("after release", after, "free MiB", free1 >> 20)
    assert after == streams0
    # the released workspaces' device memory is back (the runtime may keep a little cached)
    assert free1 >= free0 - (8 << 20), (free0, free1)
    # releasing a stream the library has no workspace for is a no-op
    zb.zero_stream_release(torch.cuda.current_stream())
    zb.zero_stream_release(torch.cuda.current_stream())
    assert all(b.guards_intact() for b in bufs)


def _record(zb, dev):
    return zb.resident_state(dev, HP["lr"], HP["beta1"], HP["beta2"], HP["eps"], HP["weight_decay"], HP["clip"],
                             2.0 ** 16, window=1000)


def test_resident_records_own_their_workspaces_under_concurrent_replays(env):
    torch, zb, dev = env
    n = 3_000_017
    cases = [workloads.random_case(5100 + i, n) for i in range(2)]
    gbufs = [_alloc(torch, dev, n) for _ in range(2)]   # replayed graphs
    ebufs = [_alloc(torch, dev, n) for _ in range(2)]   # eager resident references
    for i in range(2):
        g16, theta, m, v = cases[i]
        for bufs in (gbufs[i], ebufs[i]):
            for b, a in zip(bufs, (g16, theta, m, v, workloads.p16_sentinel(n))):
                b.upload(a)
    gstate = [_record(zb, dev) for _ in range(2)]
    estate = [_record(zb, dev) for _ in range(2)]
    # eager traffic on the capture stream uses its own arrays and record
    side = _alloc(torch, dev, n)
    for b, a in zip(side, cases[0][:4] + (workloads.p16_sentinel(n),)):
        b.upload(a)
    side_state = _record(zb, dev)
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()
    records0 = zb.zero_workspace_count()[1]
    graphs = []
    for i in range(2):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=cap):
            zb.zero_shard_step_resident(*(b.view for b in gbufs[i]), gstate[i])
        graphs.append(g)
    torch.cuda.synchronize()
    assert zb.zero_workspace_count()[1] == records0 + 2   # one workspace per captured record
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    for k in range(6):
        s1.wait_stream(torch.cuda.current_stream())
        s2.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s1):
            graphs[0].replay()
        with torch.cuda.stream(s2):
            graphs[1].replay()
        with torch.cuda.stream(cap):
            zb.zero_shard_step_resident(*(b.view for b in side), side_state)
        for i in range(2):
            zb.zero_shard_step_resident(*(b.view for b in ebufs[i]), estate[i])
        torch.cuda.synchronize()
        for i in range(2):
            a, b = zb.read_resident_state(gstate[i]), zb.read_resident_state(estate[i])
            assert bytes(a) == bytes(b) and a.t == k + 2, (k, i, a.t, b.t)
            for x, y in zip(gbufs[i][1:], ebufs[i][1:]):
                assert np.array_equal(x.download().view(np.uint8), y.download().view(np.uint8)), (k, i)
    # and the eager references follow the oracle
    g16, theta, m, v = cases[1]
    ref = [theta.copy(), m.copy(), v.copy(), workloads.p16_sentinel(n)]
    for k in range(6):
        H.oracle_step(g16, *ref, HP["lr"], HP["beta1"], HP["beta2"], HP["eps"], HP["weight_decay"], k + 1,
                      2.0 ** 16, HP["clip"])
    say("six concurrent replays", H.compare_state([b.download() for b in ebufs[1][1:]], ref))
    del graphs
    for st in gstate + estate + [side_state]:
        zb.zero_resident_release(st)
    assert zb.zero_workspace_count()[1] == records0
    assert all(b.guards_intact() for bufs in gbufs + ebufs + [side] for b in bufs)


def test_resident_record_out_of_range_is_not_a_step(env):
    torch, zb, dev = env
    n = 10_001
    g16, theta, m, v = workloads.random_case(5200, n)
    bufs = _alloc(torch, dev, n)
    for b, a in zip(bufs, (g16, theta, m, v, workloads.p16_sentinel(n))):
        b.upload(a)
    good = zb.resident_state_record(1e-4, 0.9, 0.999, 1e-8, 0.0, 1.0, 1024.0)
    for field, value in (("t", 0), ("beta1", 1.0), ("loss_scale", 0.0), ("min_scale", -1.0), ("eps", float("nan"))):
        rec = zb.ResidentState.from_buffer_copy(bytes(good))
        setattr(rec, field, value)
        state = torch.frombuffer(bytearray(bytes(rec)), dtype=torch.uint8).to(dev)
        zb.zero_shard_step_resident(*(b.view for b in bufs), state)
        torch.cuda.synchronize()
        got = zb.read_resident_state(state)
        rec.skipped = -1
        assert bytes(got) == bytes(rec), field
        for b, a in zip(bufs[1:], (theta, m, v, workloads.p16_sentinel(n))):
            assert np.array_equal(b.download().view(np.uint8), np.ascontiguousarray(a).view(np.uint8)), field
        zb.zero_resident_release(state)


def test_lamb_plan_moves_between_streams_without_waiting_for_others(env):
    torch, zb, dev = env
    n = 200_003
    seg = np.array([0, 1, 70_000, 70_003, 150_000, n], np.int64)
    g16, theta, m, v = workloads.random_case(5300, n)
    bufs = _alloc(torch, dev, n)
    for b, a in zip(bufs, (g16, theta, m, v, workloads.p16_sentinel(n))):
        b.upload(a)
    ref = [theta.copy(), m.copy(), v.copy(), workloads.p16_sentinel(n)]
    s_a, s_b, busy = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    with zb.LambPlan(seg) as plan:
        # warm the plan's work lists and the streams' workspaces
        for s in (s_a, s_b):
            assert zb.zero_lamb_step(plan, *(b.view for b in bufs), 1e-3, 0.9, 0.999, 1e-6, 0.01, 1, 2.0 ** 16,
                                     1.0, stream=s) == 0
        torch.cuda.synchronize()
        for t in (1, 1):
            H.oracle_lamb_step(g16, *ref, seg, 1e-3, 0.9, 0.999, 1e-6, 0.01, t, 2.0 ** 16, 1.0)
        with torch.cuda.stream(busy):
            torch.cuda._sleep(120_000_000)   # a bounded spin of roughly 50 ms on the third stream
        t0 = time.perf_counter()
        for k in range(6):
            s = (s_a, s_b)[k % 2]
            assert zb.zero_lamb_step(plan, *(b.view for b in bufs), 1e-3, 0.9, 0.999, 1e-6, 0.01, k + 2, 2.0 ** 16,
                                     1.0, stream=s) == 0
        host_ms = (time.perf_counter() - t0) * 1e3
        busy_done_early = busy.query()
        torch.cuda.synchronize()
        say("six alternating LAMB steps returned in %.2f ms; busy stream finished by then: %s" % (host_ms,
                                                                                                  busy_done_early))
        assert not busy_done_early and host_ms < 40.0, "the calls waited for the busy stream"
    for k in range(6):
        H.oracle_lamb_step(g16, *ref, seg, 1e-3, 0.9, 0.999, 1e-6, 0.01, k + 2, 2.0 ** 16, 1.0)
    H.compare_state([b.download() for b in bufs[1:]], ref)
    assert all(b.guards_intact() for b in bufs)


def test_lamb_probes_touch_exactly_their_arrays(env):
    torch, zb, dev = env
    n = 100_003
    g16, theta, m, v = workloads.random_case(5400, n)
    bufs = _alloc(torch, dev, n)
    for b, a in zip(bufs, (g16, theta, m, v, workloads.p16_sentinel(n))):
        b.upload(a)
    zb.zero_probe_lamb_pass(0, bufs[0].view, bufs[1].view, bufs[2].view, bufs[3].view, None)
    torch.cuda.synchronize()
    gf = g16.view(np.float16).astype(np.float32)
    assert np.array_equal(bufs[2].download(), m + gf) and np.array_equal(bufs[3].download(), v + theta)
    assert np.array_equal(bufs[1].download(), theta)
    zb.zero_probe_lamb_pass(1, None, bufs[1].view, bufs[2].view, bufs[3].view, bufs[4].view)
    torch.cuda.synchronize()
    o = (theta + (m + gf)) + (v + theta)
    assert np.array_equal(bufs[1].download(), o)
    assert np.array_equal(bufs[4].download(), o.astype(np.float16).view(np.uint16))
    assert all(b.guards_intact() for b in bufs)


def test_adam_probe_touches_exactly_its_arrays(env):
    # the update's byte-mix probe: reads the gradient and the three fp32 arrays, writes the
    # fp32 arrays and the fp16 parameters (vectors, then a 3-element tail), nothing beyond them
    torch, zb, dev = env
    n = 100_003
    g16, theta, m, v = workloads.random_case(5500, n)
    bufs = _alloc(torch, dev, n)
    for b, a in zip(bufs, (g16, theta, m, v, workloads.p16_sentinel(n))):
        b.upload(a)
    zb.zero_probe_adam_mix(*(b.view for b in bufs))
    torch.cuda.synchronize()
    gf = g16.view(np.float16).astype(np.float32)
    th = theta + gf
    assert np.array_equal(bufs[0].download(), g16)
    assert np.array_equal(bufs[1].download(), th)
    assert np.array_equal(bufs[2].download(), m + theta) and np.array_equal(bufs[3].download(), v + m)
    assert np.array_equal(bufs[4].download(), th.astype(np.float16).view(np.uint16))
    assert all(b.guards_intact() for b in bufs)
