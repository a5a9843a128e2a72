"""The allocation-free entry point (zero_shard_step_noalloc) against zero_shard_step.

Called through the C ABI twice in a row, the second time on a smaller shard, and
once more with an overflowing gradient; every result is compared with
zero_shard_step on copies of the same inputs (the same kernels: equal bit for
bit) and with the oracle (Sec. 5.1-5.2 shard step, Sec. 3.1 mixed-precision
Adam).  The library holds no more workspaces afterwards than before: the
fixed per-GPU array served every call.
"""
import ctypes
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import gpu_harness as H  # noqa: E402

from paper_1910_02054_amd import workloads  # noqa: E402

pytestmark = pytest.mark.gpu
HP = (1e-4, 0.9, 0.999, 1e-8, 0.01)


def say(*a):
    print("[gpu-noalloc]", *a, flush=True)


@pytest.fixture(scope="module")
def env():
    import torch
    from paper_1910_02054_amd import binding
    assert torch.cuda.is_available()
    return torch, binding, torch.device("cuda:0")


def _alloc(torch, dev, n):
    dts = (torch.float16, torch.float32, torch.float32, torch.float32, torch.float16)
    return [H.Guarded(torch, n, dt, dev) for dt in dts]


def _raw_step(zb, fn_name, bufs, n, t, scale, clip, stream):
    fn = getattr(zb.raw_library(), fn_name)
    return fn(*(b.view.data_ptr() for b in bufs), ctypes.c_int64(n), *HP, t, scale, clip, stream)


def test_noalloc_step_equals_the_allocating_step(env):
    torch, zb, dev = env
    stream = torch.cuda.current_stream().cuda_stream
    # warm the allocating path's workspace for this stream first, so the count below covers
    # only the allocation-free calls
    w = _alloc(torch, dev, 8)
    for buf, arr in zip(w, workloads.random_case(8799, 8)[:4] + (workloads.p16_sentinel(8),)):
        buf.upload(arr)
    assert _raw_step(zb, "zero_shard_step", w, 8, 1, 2.0 ** 16, 1.0, stream) == 0
    torch.cuda.synchronize()
    counts0 = zb.zero_workspace_count()
    for k, (n, inject) in enumerate(((3_000_017, None), (100_003, None), (40_009, 777))):
        say("call", k + 1, "n", n, "inject", inject)
        g16, theta, m, v = workloads.random_case(8800 + k, n)
        if inject is not None:
            g16[inject] = 0x7C00
        a, b = _alloc(torch, dev, n), _alloc(torch, dev, n)
        for bufs in (a, b):
            for buf, arr in zip(bufs, (g16, theta, m, v, workloads.p16_sentinel(n))):
                buf.upload(arr)
        torch.cuda.synchronize()
        rc_a = _raw_step(zb, "zero_shard_step_noalloc", a, n, 3, 2.0 ** 16, 1.0, stream)
        st_a = zb.zero_shard_last_step_stats()
        assert zb.zero_workspace_count() == counts0, "the allocation-free call created a workspace"
        rc_b = _raw_step(zb, "zero_shard_step", b, n, 3, 2.0 ** 16, 1.0, stream)
        st_b = zb.zero_shard_last_step_stats()
        torch.cuda.synchronize()
        want = 1 if inject is not None else 0
        assert rc_a == rc_b == want, (rc_a, rc_b, zb.zero_last_error())
        assert (st_a.sumsq, st_a.mult, st_a.skipped, st_a.path, st_a.n) == \
            (st_b.sumsq, st_b.mult, st_b.skipped, st_b.path, st_b.n)
        for x, y in zip(a[1:], b[1:]):
            assert np.array_equal(x.download().view(np.uint8), y.download().view(np.uint8)), k
        ref = [theta.copy(), m.copy(), v.copy(), workloads.p16_sentinel(n)]
        skip, _ = H.oracle_step(g16, *ref, *HP, 3, 2.0 ** 16, 1.0)
        assert skip == want
        say("  path", st_a.path, H.compare_state([x.download() for x in a[1:]], ref))
        assert all(buf.guards_intact() for buf in a + b)


def test_noalloc_rejects_sizes_beyond_its_limit(env):
    torch, zb, dev = env
    lib = zb.raw_library()
    G = [0x10000000, 0x20000000, 0x30000000, 0x40000000, 0x50000000]
    assert lib.zero_shard_step_noalloc(*G, (1 << 40) + 1, *HP, 1, 65536.0, 1.0, None) == zb.ZERO_EINVAL
    assert "2^40" in zb.zero_last_error()
