"""The C ABI used from a plain C99 program (tests/c_abi_driver.c): HIP's C
runtime API for memory and streams, libzeroshard for the shard step, the C
oracle for the expected bytes -- no Python or PyTorch in the process.

CPU: the program compiles warning-free against include/zero_shard.h, links the
library and the oracle, checks the host-only entry points against the oracle
(the accounting of every Table 1 cell's parameters, the bias corrections of
2000 steps) and reports that no GPU is present.  GPU: every case
(several shard lengths, aligned / equally shifted / unequally shifted arrays,
a skipped step, the split phase, a created stream and the null stream)
matches the oracle byte for byte."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def _build(tmp_path):
    import oracle
    from paper_1910_02054_amd import build as zbuild
    oracle.lib()  # builds the oracle library when it is missing
    if not os.path.exists(zbuild.LIB):
        pytest.fail("libzeroshard.so is not built")
    exe = str(tmp_path / "c_abi_driver")
    pkg, orc = os.path.dirname(zbuild.LIB), os.path.join(ROOT, "oracle")
    cmd = ["gcc", "-std=c99", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I" + os.path.join(ROCM, "include"), "-I" + os.path.join(ROOT, "include"),
           os.path.join(ROOT, "tests", "c_abi_driver.c"), "-o", exe,
           "-L" + os.path.join(ROCM, "lib"), "-lamdhip64", "-L" + pkg, "-l:libzeroshard.so",
           "-L" + orc, "-l:liboracle.so", "-Wl,-rpath," + ":".join([os.path.join(ROCM, "lib"), pkg, orc])]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, timeout=120)
    assert r.returncode == 0, r.stdout.decode(errors="replace")
    return exe


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_c_driver_builds_and_needs_a_gpu(tmp_path):
    import torch
    exe = _build(tmp_path)
    if torch.cuda.is_available():
        pytest.skip("a GPU is present: the GPU test runs the driver")
    r = subprocess.run([exe], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, timeout=60)
    out = r.stdout.decode(errors="replace")
    assert r.returncode == 77 and "host checks ok" in out, out


@pytest.mark.gpu
def test_c_driver_matches_the_oracle(tmp_path):
    exe = _build(tmp_path)
    print("[gpu-c-abi] running", exe, flush=True)
    r = subprocess.run([exe], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, timeout=100)
    out = r.stdout.decode(errors="replace")
    print(out[-2000:], flush=True)
    assert r.returncode == 0, out[-2000:]
    assert "all cases match the oracle" in out
