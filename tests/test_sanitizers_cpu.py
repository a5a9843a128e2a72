"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

* The oracle is rebuilt with gcc's ASan/UBSan and the fast oracle pins run
  against that build.
* The library's host code is rebuilt with the sanitizers applied to the host
  compilation only (the gfx950 device code is compiled as usual) and a fuzz
  driver exercises every host path that needs no GPU.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN_ENV = {"ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1", "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}


def _run(cmd, env):
    return subprocess.run(cmd, cwd=ROOT, env=dict(os.environ, **env), stdout=subprocess.PIPE,
                          stderr=subprocess.STDOUT, timeout=600)


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_asan_ubsan(tmp_path):
    lib = str(tmp_path / "liboracle_san.so")
    subprocess.run(["gcc", "-std=gnu11", "-O1", "-g", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
                    "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
                    os.path.join(ROOT, "oracle", "zero_oracle.c"), "-o", lib, "-lm"], check=True)
    rt = [subprocess.run(["gcc", "-print-file-name=" + n], stdout=subprocess.PIPE, check=True).stdout.decode().strip()
          for n in ("libasan.so", "libubsan.so")]
    r = _run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "tests/test_oracle_stats.py",
              "tests/test_oracle_adam.py", "tests/test_oracle_layout.py"],
             dict(SAN_ENV, LD_PRELOAD=" ".join(rt), ZERO_ORACLE_LIB=lib))
    assert r.returncode == 0, r.stdout.decode(errors="replace")[-3000:]


def test_library_host_code_under_asan_ubsan(tmp_path):
    from paper_1910_02054_amd import build as b
    lib = str(tmp_path / "libzeroshard_san.so")
    flags = [f for f in b.HIPCC_FLAGS if f != "-O3"] + ["-O1", "-g"]
    for s in ("address", "undefined"):
        flags += ["-Xarch_host", "-fsanitize=" + s]
    subprocess.run([b.hipcc(), *flags, *b.SOURCES, "-o", lib], check=True, stdout=subprocess.DEVNULL,
                   stderr=subprocess.DEVNULL)
    clang = os.path.join(os.path.dirname(os.path.realpath(b.hipcc())), "..", "lib", "llvm", "bin", "clang++")
    if not os.path.exists(clang):
        clang = "/opt/rocm/lib/llvm/bin/clang++"
    rt = subprocess.run([clang, "-print-file-name=libclang_rt.asan-x86_64.so"], stdout=subprocess.PIPE,
                        check=True).stdout.decode().strip()
    r = _run([sys.executable, os.path.join(ROOT, "tests", "abi_fuzz_driver.py"), lib], dict(SAN_ENV, LD_PRELOAD=rt))
    out = r.stdout.decode(errors="replace")
    assert r.returncode == 0 and "driver done" in out, out[-3000:]
