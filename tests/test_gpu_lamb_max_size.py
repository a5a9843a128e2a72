"""A LAMB shard larger than 2^31 elements (64-bit indexing in the tile walk, the
work lists and the layer sums), checked layer by layer on the layers that hold
the head, both sides of the 2^31 boundary and the tail.  A layer's trust ratio
depends on all of it, so the oracle updates each checked layer whole, with the
exact statistics of the whole gradient."""
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
B31 = 1 << 31
HP = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-6, wd=0.01)


def say(*a):
    print("[gpu-lamb-max]", *a, flush=True)


def _layer_table():
    # ~25M-element layers (odd sizes), with tiny layers and one straddling layer at 2^31
    cuts = list(range(25_165_843, B31 - 1000, 25_165_843))
    cuts += [B31 - 700, B31 - 3, B31 - 2, B31 + 1, B31 + 513, B31 + 20_000_003]
    cuts += list(range(B31 + 45_000_017, N - 1, 25_165_843))
    cuts = sorted(set(c for c in cuts if 0 < c < N))
    return np.array([0] + cuts + [N], np.int64)


def test_lamb_shard_beyond_int32_range():
    import torch
    from paper_1910_02054_amd import binding as zb
    dev = torch.device("cuda:0")
    w = workloads.WORKLOADS["gpt2_1p5b"]
    seg = _layer_table()
    say("generating", N, "elements,", seg.size - 1, "layers")
    theta, m, v = workloads.initial_state(w, N)
    g16 = workloads.gradients(w, N, 1, w.loss_scale)
    # the layers to check: first, last, and every layer within 1000 elements of 2^31
    lid = np.searchsorted(seg, [0, B31 - 1000, B31 + 1000, N - 1], side="right") - 1
    check = sorted(set([int(lid[0]), int(lid[3])] + list(range(int(lid[1]), int(lid[2]) + 1))))
    assert any(seg[k] < B31 < seg[k + 1] for k in check) or B31 in seg
    saved = {k: (g16[seg[k]:seg[k + 1]].copy(), theta[seg[k]:seg[k + 1]].copy(), m[seg[k]:seg[k + 1]].copy(),
                 v[seg[k]:seg[k + 1]].copy()) for k in check}
    say("exact statistics on the host; checking layers", check)
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
    with zb.LambPlan(seg) as plan:
        flag = zb.zero_lamb_step(plan, *d, HP["lr"], HP["beta1"], HP["beta2"], HP["eps"], HP["wd"], 1,
                                 w.loss_scale, w.clip)
        st = zb.zero_shard_last_step_stats()
        torch.cuda.synchronize()
    assert flag == 0 and abs(st.norm / sc.norm - 1) <= 1e-9
    hp = oracle.hyper(HP["lr"], HP["beta1"], HP["beta2"], HP["eps"], HP["wd"], 1)
    for k in check:
        a, b = int(seg[k]), int(seg[k + 1])
        g_s, th_s, m_s, v_s = saved[k]
        p_s = workloads.p16_sentinel(b - a)
        oracle.lamb(g_s, th_s, m_s, v_s, p_s, np.array([0, b - a], np.int64), sc.mult, hp, HP["lr"])
        got = [d[1][a:b].cpu().numpy(), d[2][a:b].cpu().numpy(), d[3][a:b].cpu().numpy(),
               d[4][a:b].view(torch.int16).cpu().numpy().view(np.uint16)]
        diag = H.compare_state(got, [th_s, m_s, v_s, p_s])
        say("layer", k, "[%d, %d)" % (a, b), diag)
    del d
    torch.cuda.empty_cache()
