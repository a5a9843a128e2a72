"""Concurrency of the host side on the GPU: seven host threads, each on its own
stream, run different entry points at the same time with sampled kernel
profiling switched on -- the fused Adam step on two streams, the split phase,
the asynchronous split phase, the resident step, and LAMB steps from two threads
that share one layer-table plan (the plan moves between their streams).  The
library serialises what shares state (a stream's workspace, a plan) and
nothing else; every thread's result must equal the oracle's (Sec. 5.1-5.2
shard step, Sec. 3.1 mixed-precision Adam; LAMB as related work in Sec. 2.3).
"""
import os
import sys
import threading

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import gpu_harness as H  # noqa: E402

from paper_1910_02054_amd import workloads  # noqa: E402

pytestmark = pytest.mark.gpu
STEPS = 4
HP = dict(lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.01, scale=2.0 ** 16, clip=1.0)


def say(*a):
    print("[gpu-concurrency]", *a, flush=True)


@pytest.fixture(scope="module")
def env():
    import torch
    from paper_1910_02054_amd import binding
    assert torch.cuda.is_available()
    return torch, binding, torch.device("cuda:0")


def _shard(torch, dev, seed, n):
    g16, theta, m, v = workloads.random_case(seed, n)
    dts = (torch.float16, torch.float32, torch.float32, torch.float32, torch.float16)
    bufs = [H.Guarded(torch, n, dt, dev) for dt in dts]
    for b, a in zip(bufs, (g16, theta, m, v, workloads.p16_sentinel(n))):
        b.upload(a)
    return bufs, g16, [theta.copy(), m.copy(), v.copy(), workloads.p16_sentinel(n)]


def test_seven_threads_on_seven_streams_with_profiling(env):
    torch, zb, dev = env
    n = 300_007
    seg = np.array([0, 1, 4, 70_001, 70_003, 150_000, n], np.int64)
    jobs = ["fused", "fused", "split", "async", "resident", "lamb_a", "lamb_b"]
    shards = [_shard(torch, dev, 1300 + k, n) for k in range(len(jobs))]
    plan = zb.LambPlan(seg)
    torch.cuda.synchronize()
    errors = []
    args = (HP["lr"], 0.9, 0.999, HP["eps"], HP["wd"])

    def work(k):
        try:
            job = jobs[k]
            bufs = shards[k][0]
            views = [b.view for b in bufs]
            s = torch.cuda.Stream()
            if job == "resident":
                state = zb.resident_state(dev, HP["lr"], 0.9, 0.999, HP["eps"], HP["wd"], HP["clip"], HP["scale"])
            if job == "async":
                d_sum = torch.zeros(1, dtype=torch.float64, device=dev)
                d_flag = torch.zeros(STEPS, dtype=torch.int32, device=dev)
            for t in range(1, STEPS + 1):
                if job == "fused":
                    assert zb.zero_shard_step(*views, *args, t, HP["scale"], HP["clip"], stream=s) == 0
                elif job == "split":
                    local = zb.zero_shard_stats(views[0], stream=s)
                    assert zb.zero_shard_apply(*views, local, *args, t, HP["scale"], HP["clip"], stream=s) == 0
                elif job == "async":
                    zb.zero_shard_stats_async(views[0], d_sum, stream=s)
                    zb.zero_shard_apply_async(*views, d_sum, *args, t, HP["scale"], HP["clip"],
                                              skipped=d_flag[t - 1:t], stream=s)
                elif job == "resident":
                    zb.zero_shard_step_resident(*views, state, stream=s)
                else:
                    assert zb.zero_lamb_step(plan, *views, HP["lr"], 0.9, 0.999, 1e-6, HP["wd"], t, HP["scale"],
                                             HP["clip"], stream=s) == 0
            s.synchronize()
            if job == "async":
                assert int(d_flag.sum().item()) == 0
            if job == "resident":
                st = zb.read_resident_state(state)
                assert st.t == STEPS + 1 and st.steps == STEPS and st.skipped == 0
        except Exception as e:  # reported below
            errors.append((jobs[k], repr(e)))

    zb.zero_profile_read()
    zb.zero_lamb_profile_read()
    zb.zero_profile_enable(2)
    try:
        threads = [threading.Thread(target=work, args=(k,)) for k in range(len(jobs))]
        say("jobs", jobs)
        for th in threads:
            th.start()
        for th in threads:
            th.join()
        torch.cuda.synchronize()
    finally:
        zb.zero_profile_enable(0)
    prof, lprof = zb.zero_profile_read(), zb.zero_lamb_profile_read()
    plan.close()
    assert not errors, errors
    say("profiled steps: adam", prof.steps, "lamb", lprof.steps)
    assert prof.steps >= 1 and lprof.steps >= 1
    for k, job in enumerate(jobs):
        bufs, g16, ref = shards[k]
        for t in range(1, STEPS + 1):
            if job.startswith("lamb"):
                H.oracle_lamb_step(g16, *ref, seg, HP["lr"], 0.9, 0.999, 1e-6, HP["wd"], t, HP["scale"], HP["clip"])
            else:
                H.oracle_step(g16, *ref, HP["lr"], 0.9, 0.999, HP["eps"], HP["wd"], t, HP["scale"], HP["clip"])
        d = H.compare_state([b.download() for b in bufs[1:]], ref)
        say(job, d)
        assert all(b.guards_intact() for b in bufs), job
