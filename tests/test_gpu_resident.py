"""GPU tests of the resident step: the whole shard step, loss scaler included,
driven by a state record in device memory (no host wait), and its capture into
a HIP graph whose replays are successive optimizer steps.

Against the oracle (Sec. 5.1-5.2 shard step, mixed-precision Adam with
dynamic loss scaling): the parameter state within the usual tolerance after
every step, the scaler's record (loss scale, t, good-step count, skip flag)
exactly; graph replays equal eager resident steps bit for bit, replay after
replay, with the program's own eager work and synchronisations between them.
"""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import gpu_harness as H  # noqa: E402

import oracle  # noqa: E402
from paper_1910_02054_amd import workloads  # noqa: E402

pytestmark = pytest.mark.gpu
HP = dict(lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01, clip=1.0)


def say(*a):
    print("[gpu-resident]", *a, flush=True)


@pytest.fixture(scope="module")
def env():
    import torch
    from paper_1910_02054_amd import binding
    assert torch.cuda.is_available()
    return torch, binding, torch.device("cuda:0")


def _alloc(torch, dev, n):
    dts = (torch.float16, torch.float32, torch.float32, torch.float32, torch.float16)
    return [H.Guarded(torch, n, dt, dev) for dt in dts]


def _grad(seed, n, scale, inject=False):
    g16 = workloads.random_case(seed, n, loss_scale=scale)[0]
    if inject:
        g16[n // 3] = 0x7C00
        g16[n // 2] = 0x7E00
    return g16


def test_resident_steps_follow_the_oracle_and_its_scaler(env):
    torch, zb, dev = env
    n = 1_000_003
    _, theta, m, v = workloads.random_case(501, n)
    bufs = _alloc(torch, dev, n)
    for b, a in zip(bufs[1:], (theta, m, v, workloads.p16_sentinel(n))):
        b.upload(a)
    window = 3
    state = zb.resident_state(dev, HP["lr"], HP["beta1"], HP["beta2"], HP["eps"], HP["weight_decay"], HP["clip"],
                              2.0 ** 16, min_scale=1.0, window=window)
    ref = [theta.copy(), m.copy(), v.copy(), workloads.p16_sentinel(n)]
    sc = oracle.Scaler(2.0 ** 16, window=window)
    for k in range(1, 11):
        scale, t = sc.scale.value, sc.t_next
        g16 = _grad(600 + k, n, scale, inject=k in (3, 7))
        bufs[0].upload(g16)
        zb.zero_shard_step_resident(*(b.view for b in bufs), state)
        torch.cuda.synchronize()
        skip, _ = H.oracle_step(g16, *ref, HP["lr"], HP["beta1"], HP["beta2"], HP["eps"], HP["weight_decay"], t,
                                scale, HP["clip"])
        sc.update(skip)
        st = zb.read_resident_state(state)
        assert (st.skipped, st.t, st.good, st.steps) == (skip, sc.t_next, sc.good.value, k), (k, st.t, st.good)
        assert st.loss_scale == sc.scale.value
        d = H.compare_state([b.download() for b in bufs[1:]], ref)
        say("step", k, "skip", skip, "scale", st.loss_scale, "t", st.t, d)
    assert all(b.guards_intact() for b in bufs)


def test_resident_graph_replays_equal_eager_steps(env):
    torch, zb, dev = env
    n = 2_000_003
    _, theta, m, v = workloads.random_case(502, n)
    graph_bufs, eager_bufs = _alloc(torch, dev, n), _alloc(torch, dev, n)
    for bufs in (graph_bufs, eager_bufs):
        for b, a in zip(bufs[1:], (theta, m, v, workloads.p16_sentinel(n))):
            b.upload(a)
    mk = lambda: zb.resident_state(dev, HP["lr"], HP["beta1"], HP["beta2"], HP["eps"], HP["weight_decay"],  # noqa
                                   HP["clip"], 2.0 ** 16, window=1000)
    st_graph, st_eager, st_warm = mk(), mk(), mk()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()
    # an eager call on the capture stream creates that stream's workspace (a scratch shard and
    # state, so the graph's own buffers start from the same state as the eager ones)
    warm = _alloc(torch, dev, n)
    with torch.cuda.stream(s):
        warm[0].view.copy_(graph_bufs[0].view)
        zb.zero_shard_step_resident(*(b.view for b in warm), st_warm)
    s.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        zb.zero_shard_step_resident(*(b.view for b in graph_bufs), st_graph)
    torch.cuda.synchronize()
    ref = [theta.copy(), m.copy(), v.copy(), workloads.p16_sentinel(n)]
    sc = oracle.Scaler(2.0 ** 16, window=1000)
    for k in range(1, 5):
        scale, t = sc.scale.value, sc.t_next
        g16 = _grad(700 + k, n, scale, inject=(k == 3))
        graph_bufs[0].upload(g16)
        eager_bufs[0].upload(g16)
        torch.cuda.synchronize()
        g.replay()                                        # the captured step, on its own stream
        zb.zero_shard_step_resident(*(b.view for b in eager_bufs), st_eager)
        torch.cuda.synchronize()
        skip, _ = H.oracle_step(g16, *ref, HP["lr"], HP["beta1"], HP["beta2"], HP["eps"], HP["weight_decay"], t,
                                scale, HP["clip"])
        sc.update(skip)
        a, b = zb.read_resident_state(st_graph), zb.read_resident_state(st_eager)
        assert bytes(a) == bytes(b) and a.t == sc.t_next and a.skipped == skip and a.loss_scale == sc.scale.value
        for x, y in zip(graph_bufs[1:], eager_bufs[1:]):
            assert np.array_equal(x.download().view(np.uint8), y.download().view(np.uint8)), k
        d = H.compare_state([x.download() for x in graph_bufs[1:]], ref)
        say("replay", k, "skip", skip, d)
    assert all(b.guards_intact() for b in graph_bufs + eager_bufs)
    del g


def test_resident_empty_shard_advances_the_scaler(env):
    torch, zb, dev = env
    state = zb.resident_state(dev, HP["lr"], HP["beta1"], HP["beta2"], HP["eps"], HP["weight_decay"], HP["clip"],
                              1024.0, window=2)
    for _ in range(3):
        zb.zero_shard_step_resident(None, None, None, None, None, state, n=0)
    torch.cuda.synchronize()
    st = zb.read_resident_state(state)
    assert (st.t, st.steps, st.skipped, st.good) == (4, 3, 0, 1) and st.loss_scale == 2048.0
