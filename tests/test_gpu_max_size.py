"""A shard larger than 2^31 elements (64-bit indexing in every kernel), checked
on sampled outputs: the oracle takes the exact statistics of the whole gradient
and then updates each sampled element one by one (the update is element-wise
given the shared scalars).  Samples cover the head, both sides of the 2^31
boundary, the tail and random positions."""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import gpu_harness as H  # noqa: E402

import oracle  # noqa: E402
from paper_1910_02054_amd import workloads  # noqa: E402

pytestmark = pytest.mark.gpu
N = (1 << 31) + (1 << 20) + 5


def say(*a):
    print("[gpu-max]", *a, flush=True)


def test_shard_beyond_int32_range():
    import torch
    from paper_1910_02054_amd import binding as zb
    dev = torch.device("cuda:0")
    w = workloads.WORKLOADS["gpt2_1p5b"]
    say("generating", N, "elements")
    theta, m, v = workloads.initial_state(w, N)
    g16 = workloads.gradients(w, N, 1, w.loss_scale)
    r = np.random.default_rng(7)
    idx = np.unique(np.concatenate([
        np.arange(0, 4096), np.arange((1 << 31) - 4096, (1 << 31) + 4096), np.arange(N - 4096, N),
        r.integers(0, N, size=200_000)])).astype(np.int64)
    samples = [a[idx].copy() for a in (g16, theta, m, v)]
    say("exact statistics on the host")
    spans = [(a, min(N, a + (1 << 24))) for a in range(0, N, 1 << 24)]
    parts = list(H._POOL.map(lambda s: oracle.local_stats(g16[s[0]:s[1]]), spans))
    sc = oracle.scalars(sum(p[0] for p in parts), max(p[1] for p in parts), w.loss_scale, w.clip)
    assert sc.skip == 0
    say("upload")
    d = [torch.from_numpy(g16.view(np.int16)).to(dev).view(torch.float16)]
    del g16
    for a in (theta, m, v):
        d.append(torch.from_numpy(a).to(dev))
    del theta, m, v
    d.append(torch.full((N,), workloads.P16_SENTINEL, dtype=torch.int16, device=dev).view(torch.float16))
    say("step")
    flag = zb.zero_shard_step(*d, w.lr, w.beta1, w.beta2, w.eps, w.weight_decay, 1, w.loss_scale, w.clip)
    st = zb.zero_shard_last_step_stats()
    torch.cuda.synchronize()
    assert flag == 0 and abs(st.norm / sc.norm - 1) <= 1e-9
    ti = torch.from_numpy(idx).to(dev)
    got = [d[k].index_select(0, ti).cpu() for k in range(1, 5)]
    got = [got[0].numpy(), got[1].numpy(), got[2].numpy(), got[3].view(torch.int16).numpy().view(np.uint16)]
    # the oracle, element by element on the samples, with the exact global multiplier
    g_s, th_s, m_s, v_s = samples
    p_s = workloads.p16_sentinel(idx.size)
    oracle.adam(g_s, th_s, m_s, v_s, p_s, sc.mult, oracle.hyper(w.lr, w.beta1, w.beta2, w.eps, w.weight_decay, 1))
    diag = H.compare_state(got, [th_s, m_s, v_s, p_s])
    diag["mult_equal"] = bool(np.float32(st.mult) == np.float32(sc.mult))
    say(diag)
    del d
    torch.cuda.empty_cache()
