"""The Python binding on the CPU: argument marshalling fails loudly (no host
fallback exists), and the LAMB plan wrapper validates layer tables before
anything reaches a device."""
import os
import subprocess
import sys
import types

import numpy as np
import pytest
import torch


@pytest.fixture(scope="module")
def zb():
    from paper_1910_02054_amd import build as b
    if b.is_stale():
        b.build()
    from paper_1910_02054_amd import binding
    return binding


def _cpu_shard(n):
    return (torch.zeros(n, dtype=torch.float16), torch.zeros(n), torch.zeros(n), torch.zeros(n),
            torch.zeros(n, dtype=torch.float16))


def test_host_tensors_are_refused(zb):
    with pytest.raises(TypeError, match="device tensor"):
        zb.zero_shard_step(*_cpu_shard(8), 1e-3, 0.9, 0.999, 1e-8, 0.0, 1, 1.0, 1.0)
    with pytest.raises(TypeError, match="device tensor"):
        zb.zero_shard_stats(torch.zeros(8, dtype=torch.float16))
    with pytest.raises(TypeError, match="device tensor"):
        zb.zero_shard_apply(*_cpu_shard(8), 1.0, 1e-3, 0.9, 0.999, 1e-8, 0.0, 1, 1.0, 1.0)


def test_wrong_dtypes_are_refused(zb):
    g, th, m, v, p = _cpu_shard(8)
    # each argument's dtype is checked before its device, in argument order
    with pytest.raises(TypeError, match="grad16: dtype"):
        zb.zero_shard_step(th, th, m, v, p, 1e-3, 0.9, 0.999, 1e-8, 0.0, 1, 1.0, 1.0)
    with pytest.raises(TypeError, match="grad16: dtype"):
        zb.zero_shard_stats(th)


def test_shard_tensors_of_different_lengths_are_refused(zb):
    g, th, m, v, p = _cpu_shard(8)
    with pytest.raises(ValueError, match="differ in length"):
        zb.zero_shard_step(g, th, m[:4], v, p, 1e-3, 0.9, 0.999, 1e-8, 0.0, 1, 1.0, 1.0)


@pytest.mark.parametrize("offs", [[0, 5, 5, 10], [1, 10], [0, 7, 3, 10]])
def test_lamb_plan_rejects_bad_tables(zb, offs):
    with pytest.raises(zb.ZeroError) as e:
        zb.LambPlan(offs)
    assert e.value.code == zb.ZERO_EINVAL


def test_lamb_plan_rejects_malformed_input(zb):
    with pytest.raises(ValueError):
        zb.LambPlan([])
    with pytest.raises(ValueError):
        zb.LambPlan(np.zeros((2, 2), np.int64))


def test_lamb_plan_needs_a_device_for_a_valid_table(zb):
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    with pytest.raises(zb.ZeroError) as e:
        zb.LambPlan([0, 10])
    assert e.value.code == zb.ZERO_EHIP


def test_lamb_wrappers_check_lengths_against_the_plan(zb):
    plan = types.SimpleNamespace(n=16, n_seg=2, handle=None)  # stands in for a plan; no call reaches C
    g, th, m, v, p = _cpu_shard(8)
    with pytest.raises(ValueError, match="plan's n"):
        zb.zero_lamb_step(plan, g, th, m, v, p, 1e-3, 0.9, 0.999, 1e-6, 0.0, 1, 1.0, 1.0)
    g, th, m, v, p = _cpu_shard(16)
    with pytest.raises(ValueError, match="2 \\* n_seg"):
        zb.zero_lamb_moments(plan, g, th, m, v, 1.0, 0.9, 0.999, 1e-6, 0.0, 1, 1.0, 1.0,
                             torch.zeros(3, dtype=torch.float64))
    with pytest.raises(TypeError, match="device tensor"):
        zb.zero_lamb_step(plan, g, th, m, v, p, 1e-3, 0.9, 0.999, 1e-6, 0.0, 1, 1.0, 1.0)


def test_exports_match_the_loaded_library(zb):
    lib = zb.raw_library()
    for name in zb.EXPORTS:
        assert hasattr(lib, name), name


def test_import_fails_loudly_without_the_library(tmp_path):
    # No fallback path exists: with the library missing, importing the binding raises.
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    code = ("import paper_1910_02054_amd.build as b; b.LIB = %r\n"
            "try:\n    import paper_1910_02054_amd.binding\nexcept ImportError as e:\n    print('refused:', e)\n"
            "else:\n    print('imported')\n" % str(tmp_path / "missing.so"))
    r = subprocess.run([sys.executable, "-c", code], cwd=root, stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                       timeout=120)
    out = r.stdout.decode(errors="replace")
    assert "refused: libzeroshard.so is not built" in out, out


def test_explicit_n_may_not_exceed_the_tensors(zb):
    # checked before any address is taken: a too-large n never reaches the library
    g, th, m, v, p = _cpu_shard(8)
    with pytest.raises(ValueError, match="exceeds a tensor of 8 elements"):
        zb.zero_shard_step(g, th, m, v, p, 1e-3, 0.9, 0.999, 1e-8, 0.0, 1, 1.0, 1.0, n=9)
    with pytest.raises(ValueError, match="exceeds"):
        zb.zero_shard_stats(g, n=100)
    with pytest.raises(ValueError, match="exceeds"):
        zb.zero_shard_apply(g, th, m, v, p, 1.0, 1e-3, 0.9, 0.999, 1e-8, 0.0, 1, 1.0, 1.0, n=9)
    with pytest.raises(ValueError, match="n is required"):
        zb.zero_shard_step(0x1000, th, m, v, p, 1e-3, 0.9, 0.999, 1e-8, 0.0, 1, 1.0, 1.0)
    with pytest.raises(ValueError, match="exceeds a buffer"):
        zb.zero_probe_copy(torch.zeros(4), torch.zeros(8), 32)


def test_prepared_step_refuses_what_the_step_refuses(zb):
    g, th, m, v, p = _cpu_shard(8)
    with pytest.raises(TypeError, match="device tensor"):
        zb.ShardStepCall([g], th, m, v, p, 1e-3, 0.9, 0.999, 1e-8, 0.0, 1.0)
    with pytest.raises(ValueError, match="at least one"):
        zb.ShardStepCall([], th, m, v, p, 1e-3, 0.9, 0.999, 1e-8, 0.0, 1.0)
    with pytest.raises(ValueError, match="differ in length"):
        zb.ShardStepCall([g, torch.zeros(9, dtype=torch.float16)], th, m, v, p, 1e-3, 0.9, 0.999, 1e-8, 0.0, 1.0)
    with pytest.raises(TypeError, match="grad16: dtype"):
        zb.ShardStepCall([g.float()], th, m, v, p, 1e-3, 0.9, 0.999, 1e-8, 0.0, 1.0)
