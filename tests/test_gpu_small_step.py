"""GPU parity of the one-launch small-shard step.

zero_shard_step takes a single cooperative launch for shards of up to 2^22
elements whose five arrays share one misalignment: the gradient statistics,
a grid barrier and the fused Adam update in one kernel (Sec. 5.1-5.2 shard
step, Sec. 3.1 mixed-precision Adam).  Checked against the oracle at every
step: lengths that select each vectors-per-thread variant, the 2^22 boundary
(2^22 + 1 takes the statistics and update kernels), every element
misalignment, a ragged tail, overflow at the first, middle and last element
(nothing written, the skip decision exact), clipping on and off, hundreds of
back-to-back steps without a host synchronisation between them (the barrier
counter's arithmetic), and steps on two streams from two threads.
"""
import os
import sys
import threading

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import gpu_harness as H  # noqa: E402

import oracle  # noqa: E402
from paper_1910_02054_amd import workloads  # noqa: E402

pytestmark = pytest.mark.gpu
HP = dict(lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.0)


def say(*a):
    print("[gpu-small]", *a, flush=True)


@pytest.fixture(scope="module")
def env():
    import torch
    from paper_1910_02054_amd import binding
    assert torch.cuda.is_available()
    return torch, binding, torch.device("cuda:0")


def _alloc(torch, dev, n, shift=0):
    dts = (torch.float16, torch.float32, torch.float32, torch.float32, torch.float16)
    return [H.Guarded(torch, n, dt, dev, shift=shift) for dt in dts]


def _run(torch, zb, dev, n, seed, steps=3, shift=0, clip=1.0, inject=None, wd=0.0, want_path=1):
    say("n", n, "seed", seed, "shift", shift, "clip", clip, "inject", inject)
    g16, theta, m, v = workloads.random_case(seed, n)
    bufs = _alloc(torch, dev, n, shift)
    for b, a in zip(bufs[1:], (theta, m, v, workloads.p16_sentinel(n))):
        b.upload(a)
    ref = [theta.copy(), m.copy(), v.copy(), workloads.p16_sentinel(n)]
    t = 1
    for k in range(steps):
        g16 = workloads.random_case(seed * 100 + k, n, loss_scale=2.0 ** 16)[0]
        if inject is not None and k == 1:
            g16[inject] = 0x7E00 if inject % 2 else 0xFC00
        bufs[0].upload(g16)
        flag = zb.zero_shard_step(*(b.view for b in bufs), HP["lr"], HP["beta1"], HP["beta2"], HP["eps"], wd, t,
                                  2.0 ** 16, clip)
        st = zb.zero_shard_last_step_stats()
        torch.cuda.synchronize()
        skip, sc = H.oracle_step(g16, *ref, HP["lr"], HP["beta1"], HP["beta2"], HP["eps"], wd, t, 2.0 ** 16, clip)
        assert flag == skip == st.skipped == st.overflow, (n, k, flag, skip)
        assert st.path == want_path, (n, st.path)
        if not skip:
            assert abs(st.norm / sc.norm - 1.0) <= 1e-9 and np.float32(st.mult) == np.float32(sc.mult)
            t += 1
        d = H.compare_state([b.download() for b in bufs[1:]], ref)
        assert all(b.guards_intact() for b in bufs)
    say("  ok", d)
    return d


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5, 7, 255, 1023, 1024, 1025, 65_537, 262_147, 1_048_576, 1_048_579,
                               2_000_001, 1 << 22])
def test_small_step_matches_the_oracle(env, n):
    torch, zb, dev = env
    _run(torch, zb, dev, n, seed=4000 + n % 997)


def test_just_above_the_threshold_takes_the_kernel_sequence(env):
    torch, zb, dev = env
    _run(torch, zb, dev, (1 << 22) + 1, seed=4100, steps=2, want_path=0)


@pytest.mark.parametrize("shift", [1, 2, 3])
def test_small_step_at_every_misalignment(env, shift):
    torch, zb, dev = env
    _run(torch, zb, dev, 100_003, seed=4200 + shift, shift=shift)


def test_unequal_misalignment_takes_the_kernel_sequence(env):
    torch, zb, dev = env
    n = 50_001
    g16, theta, m, v = workloads.random_case(4300, n)
    dts = (torch.float16, torch.float32, torch.float32, torch.float32, torch.float16)
    bufs = [H.Guarded(torch, n, dt, dev, shift=s) for dt, s in zip(dts, (0, 1, 0, 0, 0))]
    for b, a in zip(bufs, (g16, theta, m, v, workloads.p16_sentinel(n))):
        b.upload(a)
    flag = zb.zero_shard_step(*(b.view for b in bufs), HP["lr"], HP["beta1"], HP["beta2"], HP["eps"], 0.0, 1,
                              2.0 ** 16, 1.0)
    st = zb.zero_shard_last_step_stats()
    torch.cuda.synchronize()
    ref = [theta.copy(), m.copy(), v.copy(), workloads.p16_sentinel(n)]
    skip, _ = H.oracle_step(g16, *ref, HP["lr"], HP["beta1"], HP["beta2"], HP["eps"], 0.0, 1, 2.0 ** 16, 1.0)
    assert flag == skip == 0 and st.path == 0
    H.compare_state([b.download() for b in bufs[1:]], ref)


@pytest.mark.parametrize("where", ["first", "middle", "last"])
def test_small_step_overflow_writes_nothing(env, where):
    torch, zb, dev = env
    n = 300_007
    pos = {"first": 0, "middle": n // 2, "last": n - 1}[where]
    _run(torch, zb, dev, n, seed=4400 + pos % 13, inject=pos)


@pytest.mark.parametrize("clip,wd", [(0.0, 0.0), (1e6, 0.01), (1e-3, 0.1)])
def test_small_step_clipping_and_decay(env, clip, wd):
    torch, zb, dev = env
    _run(torch, zb, dev, 777_777, seed=4500, clip=clip, wd=wd)


def test_back_to_back_steps_without_synchronisation(env):
    # 300 steps queued one after another: each launch's barrier target is the counter's
    # arrivals so far plus its grid, so a miscount would deadlock-then-abort or pass early
    torch, zb, dev = env
    n, steps = 65_536 + 5, 300
    _, theta, m, v = workloads.random_case(4600, n)
    grads = [workloads.random_case(4601 + k, n)[0] for k in range(4)]
    bufs = _alloc(torch, dev, n)
    for b, a in zip(bufs[1:], (theta, m, v, workloads.p16_sentinel(n))):
        b.upload(a)
    dg = [torch.from_numpy(g.view(np.int16)).to(dev).view(torch.float16) for g in grads]
    for k in range(steps):
        assert zb.zero_shard_step(dg[k % 4], *(b.view for b in bufs[1:]), HP["lr"], HP["beta1"], HP["beta2"],
                                  HP["eps"], 0.0, k + 1, 2.0 ** 16, 1.0) == 0
    torch.cuda.synchronize()
    assert zb.zero_shard_last_step_stats().path == 1
    ref = [theta.copy(), m.copy(), v.copy(), workloads.p16_sentinel(n)]
    for k in range(steps):
        assert H.oracle_step(grads[k % 4], *ref, HP["lr"], HP["beta1"], HP["beta2"], HP["eps"], 0.0, k + 1,
                             2.0 ** 16, 1.0)[0] == 0
    d = H.compare_state([b.download() for b in bufs[1:]], ref)
    say("300 steps", d)
    assert all(b.guards_intact() for b in bufs)


def test_two_streams_two_threads(env):
    torch, zb, dev = env
    n, steps = 400_003, 40
    results, errors = {}, []

    def worker(idx):
        try:
            torch.cuda.set_device(dev)
            s = torch.cuda.Stream()
            _, theta, m, v = workloads.random_case(4700 + idx, n)
            g16 = workloads.random_case(4710 + idx, n)[0]
            with torch.cuda.stream(s):
                bufs = _alloc(torch, dev, n)
                for b, a in zip(bufs, (g16, theta, m, v, workloads.p16_sentinel(n))):
                    b.upload(a)
                for k in range(steps):
                    rc = zb.zero_shard_step(*(b.view for b in bufs), HP["lr"], HP["beta1"], HP["beta2"], HP["eps"],
                                            0.0, k + 1, 2.0 ** 16, 1.0)
                    assert rc == 0
                s.synchronize()
                results[idx] = ([b.download().copy() for b in bufs[1:]], (g16, theta, m, v))
        except Exception as e:  # reported by the main thread
            errors.append(repr(e))

    th = [threading.Thread(target=worker, args=(i,)) for i in range(2)]
    for x in th:
        x.start()
    for x in th:
        x.join()
    assert not errors, errors
    for idx in range(2):
        got, (g16, theta, m, v) = results[idx]
        ref = [theta.copy(), m.copy(), v.copy(), workloads.p16_sentinel(n)]
        for k in range(steps):
            H.oracle_step(g16, *ref, HP["lr"], HP["beta1"], HP["beta2"], HP["eps"], 0.0, k + 1, 2.0 ** 16, 1.0)
        H.compare_state(got, ref)
