"""GPU parity of the one-launch small-shard step.

zero_shard_step takes a single launch for shards small enough for one
resident grid (about 1.5 million elements on MI355X) whose five arrays share
one misalignment: the gradient statistics, a grid barrier and the fused Adam
update in one kernel (Sec. 5.1-5.2 shard step, Sec. 3.1 mixed-precision
Adam).  Checked against the oracle at every step: lengths that select each
vectors-per-thread variant (the 1,048,576-element tiny workload shard among
them), lengths past the one-launch limit (the statistics and update kernels),
every element misalignment, a ragged tail, overflow at the first, middle and
last element (nothing written, the skip decision exact), clipping on and off,
hundreds of back-to-back steps without a host synchronisation between them
(the barrier counter's arithmetic), and steps on two streams from two
threads.
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


def _run(torch, zb, dev, n, seed, steps=3, shift=0, clip=1.0, inject=None, wd=0.0, want_path=None):
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
        if want_path is not None:
            assert st.path == want_path, (n, st.path)
        if not skip:
            assert abs(st.norm / sc.norm - 1.0) <= 1e-9 and np.float32(st.mult) == np.float32(sc.mult)
            t += 1
        d = H.compare_state([b.download() for b in bufs[1:]], ref)
        assert all(b.guards_intact() for b in bufs)
    say("  ok", d)
    return d


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5, 7, 255, 1023, 1024, 1025, 65_537, 262_147, 600_001, 1_048_576,
                               1_048_579])
def test_small_step_matches_the_oracle(env, n):
    torch, zb, dev = env
    _run(torch, zb, dev, n, seed=4000 + n % 997, want_path=1)


@pytest.mark.parametrize("n", [1_300_001, 1_500_007])
def test_near_the_one_launch_limit(env, n):
    # either path, depending on the device's co-resident capacity; parity either way
    torch, zb, dev = env
    _run(torch, zb, dev, n, seed=4050 + n % 97, steps=2)


@pytest.mark.parametrize("n", [1_600_003, 2_000_001, (1 << 22) + 1])
def test_larger_shards_take_the_kernel_sequence(env, n):
    torch, zb, dev = env
    _run(torch, zb, dev, n, seed=4100 + n % 101, steps=2, want_path=0)


@pytest.mark.parametrize("shift", [1, 2, 3])
def test_small_step_at_every_misalignment(env, shift):
    torch, zb, dev = env
    _run(torch, zb, dev, 100_003, seed=4200 + shift, shift=shift, want_path=1)


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
    _run(torch, zb, dev, n, seed=4400 + pos % 13, inject=pos, want_path=1)


@pytest.mark.parametrize("clip,wd", [(0.0, 0.0), (1e6, 0.01), (1e-3, 0.1)])
def test_small_step_clipping_and_decay(env, clip, wd):
    torch, zb, dev = env
    _run(torch, zb, dev, 777_777, seed=4500, clip=clip, wd=wd, want_path=1)


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


def test_resident_small_step_replays_from_a_graph(env):
    # the resident step on a small shard is one launch whose barrier words belong to its
    # record: captured into a graph (with no eager call before) and replayed, each replay is the
    # next step, equal to eager resident steps on the same inputs and following the oracle,
    # its loss scaler included (an overflow at the third step)
    torch, zb, dev = env
    n = 500_009
    _, theta, m, v = workloads.random_case(4800, n)
    gb, eb = _alloc(torch, dev, n), _alloc(torch, dev, n)
    for bufs in (gb, eb):
        for b, a in zip(bufs[1:], (theta, m, v, workloads.p16_sentinel(n))):
            b.upload(a)
    mk = lambda: zb.resident_state(dev, HP["lr"], HP["beta1"], HP["beta2"], HP["eps"], 0.01, 1.0, 2.0 ** 16,  # noqa
                                   window=3)
    sg, se = mk(), mk()
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=cap):
        zb.zero_shard_step_resident(*(b.view for b in gb), sg)
    torch.cuda.synchronize()
    ref = [theta.copy(), m.copy(), v.copy(), workloads.p16_sentinel(n)]
    sc = oracle.Scaler(2.0 ** 16, window=3)
    for k in range(1, 8):
        scale, t = sc.scale.value, sc.t_next
        g16 = workloads.random_case(4810 + k, n, loss_scale=scale)[0]
        if k == 3:
            g16[n // 2] = 0x7C00
        gb[0].upload(g16)
        eb[0].upload(g16)
        torch.cuda.synchronize()
        g.replay()
        zb.zero_shard_step_resident(*(b.view for b in eb), se)
        torch.cuda.synchronize()
        skip, _ = H.oracle_step(g16, *ref, HP["lr"], HP["beta1"], HP["beta2"], HP["eps"], 0.01, t, scale, 1.0)
        sc.update(skip)
        a, b = zb.read_resident_state(sg), zb.read_resident_state(se)
        assert bytes(a) == bytes(b), k
        assert (a.skipped, a.t, a.good, a.steps) == (skip, sc.t_next, sc.good.value, k) and a.loss_scale == sc.scale.value
        for x, y in zip(gb[1:], eb[1:]):
            assert np.array_equal(x.download().view(np.uint8), y.download().view(np.uint8)), k
        d = H.compare_state([x.download() for x in gb[1:]], ref)
        say("resident replay", k, "skip", skip, d)
    del g
    zb.zero_resident_release(sg)
    zb.zero_resident_release(se)
    assert all(b.guards_intact() for b in gb + eb)


def test_alternating_grid_sizes_on_one_stream(env):
    # shards whose one-launch grids have 2 to 512 workgroups, stepped in turn on one stream:
    # the barrier words each launch leaves behind must serve the next launch of any size
    torch, zb, dev = env
    sizes = [4377, 1_048_576, 9, 65_537, 4377, 300_001, 1_048_576, 5]
    cases = {}
    for n in sorted(set(sizes)):
        g16, theta, m, v = workloads.random_case(4900 + n % 1000, n)
        bufs = _alloc(torch, dev, n)
        for b, a in zip(bufs, (g16, theta, m, v, workloads.p16_sentinel(n))):
            b.upload(a)
        cases[n] = (bufs, g16, [theta.copy(), m.copy(), v.copy(), workloads.p16_sentinel(n)], [1])
    for rnd in range(3):
        for n in sizes:
            bufs, g16, ref, t = cases[n]
            assert zb.zero_shard_step(*(b.view for b in bufs), HP["lr"], HP["beta1"], HP["beta2"], HP["eps"], 0.0,
                                      t[0], 2.0 ** 16, 1.0) == 0
            assert zb.zero_shard_last_step_stats().path == 1
            H.oracle_step(g16, *ref, HP["lr"], HP["beta1"], HP["beta2"], HP["eps"], 0.0, t[0], 2.0 ** 16, 1.0)
            t[0] += 1
    torch.cuda.synchronize()
    for n, (bufs, _, ref, _) in cases.items():
        H.compare_state([b.download() for b in bufs[1:]], ref)
        assert all(b.guards_intact() for b in bufs)


def test_prepared_step_call_equals_the_step(env):
    # the binding's prepared call (arrays and stream resolved once) runs the same C entry point:
    # bitwise the step's results, with two gradient buffers in turn and an overflow on the way
    torch, zb, dev = env
    n = 262_147
    _, theta, m, v = workloads.random_case(5600, n)
    grads = [workloads.random_case(5601 + k, n)[0] for k in range(2)]
    grads[1][n // 3] = 0x7E00   # the second buffer overflows
    a, b = _alloc(torch, dev, n), _alloc(torch, dev, n)
    for bufs in (a, b):
        for buf, arr in zip(bufs[1:], (theta, m, v, workloads.p16_sentinel(n))):
            buf.upload(arr)
    dg = [torch.from_numpy(g.view(np.int16)).to(dev).view(torch.float16) for g in grads]
    call = zb.ShardStepCall(dg, *(x.view for x in a[1:]), HP["lr"], HP["beta1"], HP["beta2"], HP["eps"], 0.0, 1.0)
    t = 1
    for k in range(6):
        which = 1 if k == 3 else 0
        f1 = call(t, 2.0 ** 16, which)
        f2 = zb.zero_shard_step(dg[which], *(x.view for x in b[1:]), HP["lr"], HP["beta1"], HP["beta2"], HP["eps"],
                                0.0, t, 2.0 ** 16, 1.0)
        assert f1 == f2 == (1 if which else 0)
        t += 1 - f1
    torch.cuda.synchronize()
    for x, y in zip(a[1:], b[1:]):
        assert np.array_equal(x.download().view(np.uint8), y.download().view(np.uint8))
    assert all(buf.guards_intact() for buf in a + b)


@pytest.mark.parametrize("n", [262_147, 3_000_001])
def test_scaled_step_follows_the_oracle_and_its_scaler(env, n):
    # zero_shard_step_scaled: the step at the scaler's t and loss scale, then the scaler's update, in
    # one call; against the oracle's step and scaler, with an overflow at the third step and the
    # scale growing after every two good steps (one-launch and three-kernel shards)
    torch, zb, dev = env
    _, theta, m, v = workloads.random_case(5700, n)
    grads = [workloads.random_case(5701 + k, n)[0] for k in range(2)]
    grads[1][n // 2] = 0x7C00   # the second buffer overflows
    bufs = _alloc(torch, dev, n)
    for buf, arr in zip(bufs[1:], (theta, m, v, workloads.p16_sentinel(n))):
        buf.upload(arr)
    dg = [torch.from_numpy(g.view(np.int16)).to(dev).view(torch.float16) for g in grads]
    call = zb.ShardStepCall(dg, *(x.view for x in bufs[1:]), HP["lr"], HP["beta1"], HP["beta2"], HP["eps"], 0.0, 1.0)
    sc = zb.Scaler(2.0 ** 10, window=2)
    ref_sc = oracle.Scaler(2.0 ** 10, window=2)
    ref = [theta.copy(), m.copy(), v.copy(), workloads.p16_sentinel(n)]
    for k in range(7):
        which = 1 if k == 2 else 0
        say("scaled step %d of n=%d (buffer %d)" % (k, n, which))
        flag = call.scaled(sc, which)
        skip, _ = H.oracle_step(grads[which], *ref, HP["lr"], HP["beta1"], HP["beta2"], HP["eps"], 0.0,
                                ref_sc.t_next, ref_sc.scale.value, 1.0)
        ref_sc.update(skip)
        assert flag == skip == (1 if which else 0)
        assert (sc.state.scale, sc.state.applied, sc.state.good) == \
            (ref_sc.scale.value, ref_sc.applied.value, ref_sc.good.value)
        assert zb.zero_shard_last_step_stats().path == (1 if n < 1_000_000 else 0)
    torch.cuda.synchronize()
    H.compare_state([b.download() for b in bufs[1:]], ref)
    assert all(b.guards_intact() for b in bufs)
