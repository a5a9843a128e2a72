"""The resident step's fp32 constants equal the eager step's, bit for bit.

Both derive the bias corrections 1 - beta^t from one definition (the power
rounded to double, the difference rounded once to fp32), the eager calls on
the host and the resident step on the device.  One-element shards make each
step's result a direct function of the constants: with lr = 1 and theta = 0
the new parameter is minus Adam's direction u = (m / bc1) / (sqrt(v / bc2) +
eps), so a one-ulp change in a bias correction shows in the output.  For
beta1 in {0.9, 0.95}, beta2 in {0.98, 0.999, 0.9999} and t = 1 .. 20,000,
element t-1 of the arrays takes the step with that t, through the resident
step (its record's t advancing on the device) and through zero_shard_step;
the two results are compared bitwise, and with the oracle.
"""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))

import oracle  # noqa: E402

pytestmark = pytest.mark.gpu
T_MAX = 20_000


def say(*a):
    print("[gpu-bias-sweep]", *a, flush=True)


@pytest.fixture(scope="module")
def env():
    import torch
    from paper_1910_02054_amd import binding
    assert torch.cuda.is_available()
    return torch, binding, torch.device("cuda:0")


@pytest.mark.parametrize("beta1", [0.9, 0.95])
def test_resident_constants_equal_eager_constants(env, beta1):
    torch, zb, dev = env
    n = T_MAX
    g16 = np.full(n, 0x3C00, np.uint16)               # 1.0 at loss scale 1
    zeros = np.zeros(n, np.float32)
    for beta2 in (0.98, 0.999, 0.9999):
        say("beta1", beta1, "beta2", beta2)
        dev_arrays = []
        for _ in range(2):
            g = torch.from_numpy(g16.view(np.int16)).to(dev).view(torch.float16)
            th, m, v = (torch.zeros(n, dtype=torch.float32, device=dev) for _ in range(3))
            p = torch.zeros(n, dtype=torch.float16, device=dev)
            dev_arrays.append((g, th, m, v, p))
        state = zb.resident_state(dev, 1.0, beta1, beta2, 1e-8, 0.0, 0.0, 1.0, window=0)
        res, eag = dev_arrays
        for t in range(1, T_MAX + 1):
            i = t - 1
            zb.zero_shard_step_resident(*(a[i:i + 1] for a in res), state)
            assert zb.zero_shard_step(*(a[i:i + 1] for a in eag), 1.0, beta1, beta2, 1e-8, 0.0, t, 1.0, 0.0) == 0
        torch.cuda.synchronize()
        rec = zb.read_resident_state(state)
        assert rec.t == T_MAX + 1 and rec.steps == T_MAX
        got_r = [a.cpu().numpy().view(np.uint8) for a in res[1:]]
        got_e = [a.cpu().numpy().view(np.uint8) for a in eag[1:]]
        for x, y, name in zip(got_r, got_e, ("master", "m", "v", "p16")):
            bad = np.flatnonzero(x.reshape(n, -1).any(axis=1) != y.reshape(n, -1).any(axis=1)) if False else None
            assert np.array_equal(x, y), "%s differs between the resident and the eager step" % name
        # the oracle, element by element: one step from zero state with that t
        th_o, m_o, v_o = zeros.copy(), zeros.copy(), zeros.copy()
        p_o = np.zeros(n, np.uint16)
        for t in range(1, T_MAX + 1):
            i = t - 1
            oracle.shard_step(g16[i:i + 1], th_o[i:i + 1], m_o[i:i + 1], v_o[i:i + 1], p_o[i:i + 1], 1.0, beta1,
                              beta2, 1e-8, 0.0, t, 1.0, 0.0)
        assert np.array_equal(got_e[0], th_o.view(np.uint8)) and np.array_equal(got_e[3], p_o.view(np.uint8))
        zb.zero_resident_release(state)
