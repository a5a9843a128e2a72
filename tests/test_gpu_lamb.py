"""GPU parity of the LAMB shard step (the C ABI's zero_lamb_* calls) against the
CPU oracle's LAMB (exact layer norms).

LAMB (You et al.) is one of the adaptive optimizers ZeRO's related work
(Sec. 2.3) lists as made affordable by partitioning optimizer state.  Layer
tables come from GPT-2-like shapes of ZeRO's evaluation (Sec. 10), cut at the
rank's shard; small and ragged tables cover layers of 1..3 elements, layers
that cross tiles, misaligned views and the scalar path.  The bar is the Adam
path's: master/m/v within max|d| <= 1e-6 * max(1, |x|), fp16 within 1 ulp,
skip flags and loss-scale sequence exact, guard canaries intact.
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
LAMB_HP = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-6, wd=0.01)


def say(*a):
    print("[gpu-lamb]", *a, flush=True)


@pytest.fixture(scope="module")
def env():
    import torch
    from paper_1910_02054_amd import binding
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch, binding, torch.device("cuda:0")


def _alloc(torch, dev, n, shifts=(0, 0, 0, 0, 0)):
    dts = (torch.float16, torch.float32, torch.float32, torch.float32, torch.float16)
    return [H.Guarded(torch, n, dt, dev, sh) for dt, sh in zip(dts, shifts)]


def _check_step(env, plan, bufs, ref, g16, seg, hp, t, scale, clip, phi=(0.0, float("inf")), label=""):
    torch, zb, dev = env
    bufs[0].upload(g16)
    flag = zb.zero_lamb_step(plan, *(b.view for b in bufs), hp["lr"], hp["beta1"], hp["beta2"], hp["eps"],
                             hp["wd"], t, scale, clip, phi[0], phi[1])
    st = zb.zero_shard_last_step_stats()
    torch.cuda.synchronize()
    skip, sc, _ = H.oracle_lamb_step(g16, *ref, seg, hp["lr"], hp["beta1"], hp["beta2"], hp["eps"], hp["wd"], t,
                                     scale, clip, phi[0], phi[1])
    assert flag == skip and st.skipped == skip, (label, flag, skip)
    d = H.compare_state([b.download() for b in bufs[1:]], ref)
    if not skip:
        assert abs(st.norm / sc.norm - 1.0) <= 1e-9
        d["mult_equal"] = bool(np.float32(st.mult) == np.float32(sc.mult))
    assert all(b.guards_intact() for b in bufs), "guard canaries overwritten"
    return flag, d


def _run_case(env, seg, g16_steps, theta, m, v, hp=LAMB_HP, scale=2.0 ** 16, clip=1.0, shifts=(0,) * 5,
              phi=(0.0, float("inf")), label=""):
    torch, zb, dev = env
    seg = np.asarray(seg, np.int64)
    n = int(seg[-1])
    bufs = _alloc(torch, dev, n, shifts)
    for b, a in zip(bufs[1:4], (theta, m, v)):
        b.upload(a)
    bufs[4].upload(workloads.p16_sentinel(n))
    ref = [theta.copy(), m.copy(), v.copy(), workloads.p16_sentinel(n)]
    out = []
    with zb.LambPlan(seg) as plan:
        for k, g16 in enumerate(g16_steps):
            say(label, "step", k + 1, "n", n, "layers", seg.size - 1, "shifts", shifts)
            out.append(_check_step(env, plan, bufs, ref, g16, seg, hp, k + 1, scale, clip, phi, label))
    return out, bufs, ref


@pytest.mark.parametrize("key,steps", [("tiny", 3), ("gpt2_1p5b", 2), ("mp16_dp25_100b", 2), ("ragged_1t", 8)])
def test_lamb_workload_shards(env, key, steps):
    torch, zb, dev = env
    w = workloads.WORKLOADS[key]
    lay = zb.zero_partition_layout(w.psi, w.nd, w.rank)
    n = lay.valid_numel
    sizes = workloads.model_tensor_sizes(workloads.MODEL_SHAPES[key], w.psi)
    seg = workloads.layer_offsets_in(sizes, lay.offset, lay.offset + n)
    theta, m, v = workloads.initial_state(w, n)
    shift = lay.offset % 8
    bufs = _alloc(torch, dev, n, (shift,) * 5)
    for b, a in zip(bufs[1:4], (theta, m, v)):
        b.upload(a)
    bufs[4].upload(workloads.p16_sentinel(n))
    ref = [theta, m, v, workloads.p16_sentinel(n)]
    s_gpu, s_ora = zb.Scaler(w.loss_scale), oracle.Scaler(w.loss_scale)
    say(key, "n", n, "layers", seg.size - 1, "offset mod 8", shift)
    with zb.LambPlan(seg) as plan:
        for step in range(1, steps + 1):
            assert s_gpu.scale == s_ora.scale.value and s_gpu.t_next == s_ora.t_next
            scale, t = s_gpu.scale, s_gpu.t_next
            g16 = workloads.gradients(w, n, step, scale)
            say(key, "step", step, "t", t, "scale", scale)
            flag, d = _check_step(env, plan, bufs, ref, g16, seg, LAMB_HP, t, scale, w.clip, label=key)
            s_gpu.update(flag)
            s_ora.update(flag)
            say(key, "step", step, "skip", flag, d)
    if w.inject_steps:
        assert s_gpu.t_next == steps + 1 - sum(1 for s in w.inject_steps if s <= steps)


def _random_layers(rng, n, small=False):
    if n < 2:
        return np.array([0, n], np.int64)
    if small:
        cuts = np.unique(np.concatenate([[1, 2, 3, 5, 8, 255, 256, 257, 300, 511, 513],
                                         rng.integers(1, n, size=max(1, n // 97))]))
    else:
        cuts = np.unique(rng.integers(1, n, size=max(1, n // 5000)))
    cuts = cuts[(cuts > 0) & (cuts < n)]
    return np.concatenate([[0], cuts, [n]]).astype(np.int64)


@pytest.mark.parametrize("n,small,shifts", [
    (1, False, (0,) * 5),
    (3, False, (1,) * 5),
    (4099, True, (0,) * 5),
    (4099, True, (1,) * 5),
    (4099, True, (2,) * 5),
    (4099, True, (3,) * 5),
    (100_003, True, (0,) * 5),
    (100_003, False, (3,) * 5),
    (100_003, True, (0, 1, 2, 3, 0)),   # mixed misalignment: scalar path
    (1_000_003, False, (1,) * 5),
])
def test_lamb_random_layer_tables(env, n, small, shifts):
    rng = np.random.default_rng(n + 7 * sum(shifts) + small)
    seg = _random_layers(rng, n, small)
    g16, theta, m, v = workloads.random_case(300 + n, n)
    g2 = workloads.random_case(301 + n, n)[0]
    _run_case(env, seg, [g16, g2], theta, m, v, shifts=shifts, label="random-%d" % n)


def test_lamb_hyperparameters_and_phi(env):
    n = 50_000
    g16, theta, m, v = workloads.random_case(401, n)
    seg = [0, 17, 4096, 30_000, n]
    for hp, phi, clip in ((dict(LAMB_HP, wd=0.0), (0.0, float("inf")), 1.0),
                          (dict(LAMB_HP, lr=0.05, wd=0.1), (0.0, 0.5), 0.0),
                          (dict(LAMB_HP, beta1=0.0, eps=1e-8), (2.0, 10.0), 1e-3),
                          (dict(LAMB_HP, lr=0.0), (0.0, float("inf")), 1.0)):
        _run_case(env, seg, [g16], theta, m, v, hp=hp, clip=clip, phi=phi, label="hp")


def test_lamb_zero_layers_and_zero_gradient(env):
    n = 20_000
    g16, theta, m, v = workloads.random_case(402, n, warm=False)
    theta[5000:6000] = 0.0          # a zero layer: trust ratio 1
    g16[12000:13000] = 0            # zero gradient with zero state: u = wd*theta
    seg = [0, 5000, 6000, 12000, 13000, n]
    _run_case(env, seg, [g16], theta, m, v, label="zero-layers")


@pytest.mark.parametrize("where", [0, 9999, 19_999])
def test_lamb_overflow_skips_without_writing(env, where):
    torch, zb, dev = env
    n = 20_000
    g16, theta, m, v = workloads.random_case(403, n)
    g16[where] = 0x7E00
    res, bufs, ref = _run_case(env, [0, 7000, n], [g16], theta, m, v, label="overflow")
    assert res[0][0] == 1
    assert np.array_equal(bufs[1].download(), theta) and np.array_equal(bufs[2].download(), m)
    assert np.array_equal(bufs[3].download(), v) and np.all(bufs[4].download() == workloads.P16_SENTINEL)


def test_lamb_deterministic(env):
    torch, zb, dev = env
    n = 1_000_003
    rng = np.random.default_rng(5)
    seg = _random_layers(rng, n)
    g16, theta, m, v = workloads.random_case(404, n)
    outs = []
    for rep in range(2):
        _, bufs, _ = _run_case(env, seg, [g16], theta, m, v, label="det-%d" % rep)
        outs.append([b.download().copy() for b in bufs[1:]])
    for a, b in zip(*outs):
        assert np.array_equal(a.view(np.uint8), b.view(np.uint8))


@pytest.mark.parametrize("psi,nd", [(4_194_304, 4), (1_000_003, 7), (333_331, 13), (2_000_001, 3)])
def test_lamb_split_phase_layers_across_shards(env, psi, nd):
    # N_d ranks emulated on one GPU; the model's layers straddle shard boundaries, so each
    # rank's boundary layers need the neighbours' partial sums (exchanged here in rank order)
    torch, zb, dev = env
    w = workloads.WORKLOADS["tiny"]
    sizes = workloads.model_tensor_sizes(workloads.MODEL_SHAPES["tiny"], psi)
    theta, m, v = workloads.initial_state(w, psi)
    m += np.float32(1e-5)
    v += np.float32(1e-9)
    ref = [theta.copy(), m.copy(), v.copy(), workloads.p16_sentinel(psi)]
    glob = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    dev_state = [torch.from_numpy(a.copy()).to(dev) for a in (theta, m, v)]
    p16 = torch.full((psi,), workloads.P16_SENTINEL, dtype=torch.int16, device=dev).view(torch.float16)
    g_dev = torch.empty(psi, dtype=torch.float16, device=dev)
    ranks = []
    for r in range(nd):
        lay = zb.zero_partition_layout(psi, nd, r)
        a, b = lay.offset, lay.offset + lay.valid_numel
        seg = workloads.layer_offsets_in(sizes, a, b)
        ranks.append(dict(a=a, b=b, seg=seg, ids=workloads.layer_ids_in(sizes, a, b), plan=zb.LambPlan(seg),
                          sums=torch.zeros(2 * (seg.size - 1), dtype=torch.float64, device=dev)))
    hp = LAMB_HP
    try:
        for t in range(1, 4):
            g16 = workloads.gradients(w, psi, t, w.loss_scale)
            g_dev.copy_(torch.from_numpy(g16.view(np.int16)).view(torch.float16))
            local = [zb.zero_shard_stats(g_dev[rk["a"]:rk["b"]]) for rk in ranks]
            gsum = 0.0
            for x in local:
                gsum += x
            for rk in ranks:
                sl = slice(rk["a"], rk["b"])
                assert zb.zero_lamb_moments(rk["plan"], g_dev[sl], dev_state[0][sl], dev_state[1][sl],
                                            dev_state[2][sl], gsum, hp["beta1"], hp["beta2"], hp["eps"], hp["wd"], t,
                                            w.loss_scale, w.clip, rk["sums"]) == 0
            # exchange: every layer's total over the ranks that hold a piece of it, in rank order
            host = [rk["sums"].cpu().numpy().reshape(-1, 2) for rk in ranks]
            total = {}
            for rk, h in zip(ranks, host):
                for gid, row in zip(rk["ids"], h):
                    acc = total.get(int(gid), (0.0, 0.0))
                    total[int(gid)] = (acc[0] + row[0], acc[1] + row[1])
            for rk in ranks:
                full = np.array([total[int(g)] for g in rk["ids"]], np.float64).reshape(-1)
                rk["sums"].copy_(torch.from_numpy(full))
            for rk in ranks:
                sl = slice(rk["a"], rk["b"])
                assert zb.zero_lamb_apply(rk["plan"], dev_state[0][sl], dev_state[1][sl], dev_state[2][sl], p16[sl],
                                          gsum, rk["sums"], hp["lr"], hp["beta1"], hp["beta2"], hp["eps"], hp["wd"],
                                          t) == 0
            torch.cuda.synchronize()
            skip, sc, per_layer = H.oracle_lamb_step(g16, *ref, glob, hp["lr"], hp["beta1"], hp["beta2"], hp["eps"],
                                                     hp["wd"], t, w.loss_scale, w.clip)
            assert skip == 0 and abs(gsum / sc.sumsq - 1) <= 1e-12
            # the exchanged layer sums against the oracle's exact ones
            for gid, (ws, us) in total.items():
                assert abs(ws / per_layer[gid, 0] - 1) <= 1e-12 and abs(us / per_layer[gid, 1] - 1) <= 1e-12
            gpu = [x.cpu().numpy() for x in dev_state] + [p16.view(torch.int16).cpu().numpy().view(np.uint16)]
            d = H.compare_state(gpu, ref)
            say("split psi", psi, "nd", nd, "step", t, d)
    finally:
        for rk in ranks:
            rk["plan"].close()


def test_lamb_split_phase_skip_and_argument_errors(env):
    torch, zb, dev = env
    n = 1000
    g16, theta, m, v = workloads.random_case(405, n)
    bufs = _alloc(torch, dev, n)
    for b, a in zip(bufs, (g16, theta, m, v, workloads.p16_sentinel(n))):
        b.upload(a)
    sums = torch.zeros(4, dtype=torch.float64, device=dev)
    with zb.LambPlan([0, 400, n]) as plan:
        hp = LAMB_HP
        assert zb.zero_lamb_moments(plan, bufs[0].view, bufs[1].view, bufs[2].view, bufs[3].view, float("inf"),
                                    hp["beta1"], hp["beta2"], hp["eps"], hp["wd"], 1, 1.0, 1.0, sums) == 1
        assert zb.zero_lamb_apply(plan, bufs[1].view, bufs[2].view, bufs[3].view, bufs[4].view, float("inf"), sums,
                                  hp["lr"], hp["beta1"], hp["beta2"], hp["eps"], hp["wd"], 1) == 1
        torch.cuda.synchronize()
        assert np.array_equal(bufs[2].download(), m) and np.all(bufs[4].download() == workloads.P16_SENTINEL)
        with pytest.raises(ValueError):     # layer sums of the wrong length
            zb.zero_lamb_moments(plan, bufs[0].view, bufs[1].view, bufs[2].view, bufs[3].view, 1.0, hp["beta1"],
                                 hp["beta2"], hp["eps"], hp["wd"], 1, 1.0, 1.0, sums[:2])
        with pytest.raises(ValueError):      # shard of the wrong length
            zb.zero_lamb_step(plan, bufs[0].view[:10], bufs[1].view[:10], bufs[2].view[:10], bufs[3].view[:10],
                              bufs[4].view[:10], 1e-3, 0.9, 0.999, 1e-6, 0.0, 1, 1.0, 1.0)
        with pytest.raises(zb.ZeroError) as e:   # phi_hi below phi_lo
            zb.zero_lamb_step(plan, *(b.view for b in bufs), 1e-3, 0.9, 0.999, 1e-6, 0.0, 1, 1.0, 1.0, 2.0, 1.0)
        assert e.value.code == zb.ZERO_EINVAL
        with pytest.raises(zb.ZeroError) as e:   # arrays overlap
            zb.zero_lamb_step(plan, bufs[0].view, bufs[1].view, bufs[1].view, bufs[3].view, bufs[4].view, 1e-3, 0.9,
                              0.999, 1e-6, 0.0, 1, 1.0, 1.0)
        assert e.value.code == zb.ZERO_EINVAL
    assert all(b.guards_intact() for b in bufs)


def test_lamb_plan_on_two_streams(env):
    # a plan used on a second stream waits for the first stream's work
    torch, zb, dev = env
    n = 300_001
    rng = np.random.default_rng(9)
    seg = _random_layers(rng, n)
    g16, theta, m, v = workloads.random_case(406, n)
    ref = [theta.copy(), m.copy(), v.copy(), workloads.p16_sentinel(n)]
    bufs = _alloc(torch, dev, n)
    for b, a in zip(bufs, (g16, theta, m, v, workloads.p16_sentinel(n))):
        b.upload(a)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    hp = LAMB_HP
    with zb.LambPlan(seg) as plan:
        for t, s in ((1, s1), (2, s2), (3, s1)):
            assert zb.zero_lamb_step(plan, *(b.view for b in bufs), hp["lr"], hp["beta1"], hp["beta2"], hp["eps"],
                                     hp["wd"], t, 2.0 ** 16, 1.0, stream=s) == 0
            s.synchronize()
            skip, _, _ = H.oracle_lamb_step(g16, *ref, seg, hp["lr"], hp["beta1"], hp["beta2"], hp["eps"], hp["wd"],
                                            t, 2.0 ** 16, 1.0)
            assert skip == 0
    torch.cuda.synchronize()
    d = H.compare_state([b.download() for b in bufs[1:]], ref)
    say("two streams", d)


def test_lamb_sampled_profile(env):
    torch, zb, dev = env
    n = 2_000_000
    rng = np.random.default_rng(11)
    seg = _random_layers(rng, n)
    g16, theta, m, v = workloads.random_case(407, n)
    bufs = _alloc(torch, dev, n)
    for b, a in zip(bufs, (g16, theta, m, v, workloads.p16_sentinel(n))):
        b.upload(a)
    zb.zero_lamb_profile_read()
    zb.zero_profile_enable(2)
    try:
        with zb.LambPlan(seg) as plan:
            for t in range(1, 7):
                zb.zero_lamb_step(plan, *(b.view for b in bufs), 1e-3, 0.9, 0.999, 1e-6, 0.0, t, 2.0 ** 16, 1.0)
        p = zb.zero_lamb_profile_read()
    finally:
        zb.zero_profile_enable(0)
    assert p.steps == 3 and p.moments_ms > 0 and p.apply_ms > 0 and p.layer_ms > 0 and p.stats_ms > 0
    say("profile", p.steps, p.stats_ms, p.moments_ms, p.layer_ms, p.apply_ms)
