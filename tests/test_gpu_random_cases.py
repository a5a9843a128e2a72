"""Seeded randomized differential tests on the GPU.

Many small shard steps with random lengths (0 to 300,000), array alignments
(equal shifts: vector path with a head; unequal shifts: scalar path), Adam
hyperparameters (lr including 0, beta1 and beta2 including 0, eps, decoupled
weight decay), step t, loss scales (powers of two and not), clip thresholds
(off, binding, never reached), warm or cold moments and injected inf/NaN
gradients.  Every case runs through the fused step, the synchronous split
phase, the asynchronous split phase and the resident step (each on its own
copy of the state) and is compared with the oracle (Sec. 5.1-5.2 shard step,
Sec. 3.1 mixed-precision Adam); LAMB steps over random layer tables with
random trust-ratio bounds likewise.  Every case is a valid input.  Each case
prints its seed, so it can be replayed.
"""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import gpu_harness as H  # noqa: E402

from paper_1910_02054_amd import workloads  # noqa: E402

pytestmark = pytest.mark.gpu
N_CASES = 48
PATHS = ("fused", "split", "async", "resident")


def say(*a):
    print("[gpu-random]", *a, flush=True)


@pytest.fixture(scope="module")
def env():
    import torch
    from paper_1910_02054_amd import binding
    assert torch.cuda.is_available()
    return torch, binding, torch.device("cuda:0")


def _draw(seed):
    r = np.random.default_rng([20191002, seed])
    kind = int(r.integers(0, 3))
    n = int((r.integers(0, 64), r.integers(64, 5000), r.integers(5000, 300_000))[kind])
    if r.random() < 0.6:
        shifts = (int(r.integers(0, 8)),) * 5
    else:
        shifts = tuple(int(x) for x in r.integers(0, 8, 5))
    hp = dict(lr=0.0 if r.random() < 0.05 else float(10.0 ** r.uniform(-6, -2)),
              beta1=float(r.choice([0.0, 0.5, 0.9, 0.95])), beta2=float(r.choice([0.0, 0.98, 0.999, 0.9999])),
              eps=float(r.choice([1e-12, 1e-8, 1e-6])), wd=float(r.choice([0.0, 0.0, 0.01, 0.1])),
              t=int(r.integers(1, 5000)),
              scale=float(2.0 ** int(r.integers(0, 17))) * (0.75 if r.random() < 0.2 else 1.0),
              clip=float(r.choice([-1.0, 0.0, 1e-3, 1.0, 1e6])))
    grad_std = float(10.0 ** r.uniform(-5, -2))
    warm = bool(r.random() < 0.7)
    inject = None
    if n > 0 and r.random() < 0.15:
        inject = (int(r.integers(0, n)), int(r.choice([0x7C00, 0xFC00, 0x7E00, 0x7C01])))
    return n, shifts, hp, grad_std, warm, inject


def _bufs(torch, dev, n, shifts):
    dts = (torch.float16, torch.float32, torch.float32, torch.float32, torch.float16)
    return [H.Guarded(torch, n, dt, dev, shift=s) for dt, s in zip(dts, shifts)]


@pytest.mark.parametrize("seed", range(N_CASES))
def test_random_adam_case_through_every_path(env, seed):
    torch, zb, dev = env
    n, shifts, hp, grad_std, warm, inject = _draw(seed)
    say("seed", seed, "n", n, "shifts", shifts, hp, "std %.2g" % grad_std, "warm", warm, "inject", inject)
    g16, theta, m, v = workloads.random_case(7000 + seed, n, grad_std=grad_std, loss_scale=hp["scale"], warm=warm)
    if inject:
        g16[inject[0]] = inject[1]
    ref = [theta.copy(), m.copy(), v.copy(), workloads.p16_sentinel(n)]
    skip, sc = H.oracle_step(g16, *ref, hp["lr"], hp["beta1"], hp["beta2"], hp["eps"], hp["wd"], hp["t"],
                             hp["scale"], hp["clip"])
    assert skip == (1 if inject else 0)
    args = (hp["lr"], hp["beta1"], hp["beta2"], hp["eps"], hp["wd"], hp["t"], hp["scale"], hp["clip"])
    for path in PATHS:
        bufs = _bufs(torch, dev, n, shifts)
        for b, a in zip(bufs, (g16, theta, m, v, workloads.p16_sentinel(n))):
            b.upload(a)
        views = [b.view for b in bufs]
        if path == "fused":
            flag = zb.zero_shard_step(*views, *args)
        elif path == "split":
            local = zb.zero_shard_stats(views[0])
            flag = zb.zero_shard_apply(*views, local, *args)
        elif path == "async":
            d_sum = torch.zeros(1, dtype=torch.float64, device=dev)
            d_flag = torch.full((1,), -1, dtype=torch.int32, device=dev)
            zb.zero_shard_stats_async(views[0], d_sum)
            zb.zero_shard_apply_async(*views, d_sum, *args, skipped=d_flag)
            torch.cuda.synchronize()
            flag = int(d_flag.item())
        else:
            state = zb.resident_state(dev, hp["lr"], hp["beta1"], hp["beta2"], hp["eps"], hp["wd"], hp["clip"],
                                      hp["scale"], window=1000, t=hp["t"])
            zb.zero_shard_step_resident(*views, state)
            torch.cuda.synchronize()
            st = zb.read_resident_state(state)
            flag = st.skipped
            assert st.t == hp["t"] + (0 if skip else 1) and st.steps == 1
            assert st.loss_scale == (max(hp["scale"] / 2, 1.0) if skip else hp["scale"])
        torch.cuda.synchronize()
        assert flag == skip, (path, flag, skip)
        d = H.compare_state([b.download() for b in bufs[1:]], ref)
        assert all(b.guards_intact() for b in bufs), path
        if any(d.get(k) for k in ("master_bitdiff", "m_bitdiff", "v_bitdiff", "p16_bitdiff")):
            say("  ", path, d)


def _random_table(r, n):
    if n == 0:
        return np.array([0], np.int64)
    cuts = set()
    for _ in range(int(r.integers(0, 12))):
        cuts.add(int(r.integers(1, n)) if n > 1 else 1)
    for _ in range(int(r.integers(0, 4))):           # a few very small layers
        a = int(r.integers(1, max(2, n - 3)))
        cuts.update({a, a + 1, a + 3})
    cuts = sorted(c for c in cuts if 0 < c < n)
    return np.array([0] + cuts + [n], np.int64)


@pytest.mark.parametrize("seed", range(16))
def test_random_lamb_case(env, seed):
    torch, zb, dev = env
    r = np.random.default_rng([1904, seed])
    n = int(r.integers(1, 200_000))
    seg = _random_table(r, n)
    shifts = (int(r.integers(0, 8)),) * 5 if r.random() < 0.6 else tuple(int(x) for x in r.integers(0, 8, 5))
    lr, b1, b2 = float(10.0 ** r.uniform(-5, -2)), float(r.choice([0.0, 0.9])), float(r.choice([0.99, 0.999]))
    eps, wd, t = float(r.choice([1e-8, 1e-6])), float(r.choice([0.0, 0.01])), int(r.integers(1, 100))
    scale, clip = float(2.0 ** int(r.integers(4, 17))), float(r.choice([0.0, 1e-3, 1.0]))
    phi_lo, phi_hi = (0.0, float("inf")) if r.random() < 0.5 else (float(r.uniform(0, 0.01)), float(r.uniform(0.05, 10)))
    say("lamb seed", seed, "n", n, "layers", seg.size - 1, "shifts", shifts, "phi", (phi_lo, phi_hi), "clip", clip)
    g16, theta, m, v = workloads.random_case(9000 + seed, n, grad_std=1e-3, loss_scale=scale, warm=True)
    ref = [theta.copy(), m.copy(), v.copy(), workloads.p16_sentinel(n)]
    skip, _, _ = H.oracle_lamb_step(g16, *ref, seg, lr, b1, b2, eps, wd, t, scale, clip, phi_lo, phi_hi)
    bufs = _bufs(torch, dev, n, shifts)
    for b, a in zip(bufs, (g16, theta, m, v, workloads.p16_sentinel(n))):
        b.upload(a)
    with zb.LambPlan(seg) as plan:
        flag = zb.zero_lamb_step(plan, *(b.view for b in bufs), lr, b1, b2, eps, wd, t, scale, clip, phi_lo, phi_hi)
        torch.cuda.synchronize()
    assert flag == skip == 0
    d = H.compare_state([b.download() for b in bufs[1:]], ref)
    assert all(b.guards_intact() for b in bufs)
    if any(d.get(k) for k in ("master_bitdiff", "m_bitdiff", "v_bitdiff", "p16_bitdiff")):
        say("  lamb", d)
