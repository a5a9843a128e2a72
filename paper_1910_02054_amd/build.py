"""Build ``libzeroshard.so`` for gfx950 with hipcc (cross-compiles without a GPU).

Flags that matter for the numerics: ``-ffp-contract=off`` keeps every fp32
multiply and add separately rounded; HIP's default correctly rounded fp32
division and square root and its default fp32/fp16 denormal handling are kept
(no fast-math).  Packed fp32 instructions are disabled.
"""
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
SOURCES = [os.path.join(CSRC, "zero_shard.hip"), os.path.join(CSRC, "zero_lamb.hip")]
DEPS = SOURCES + [os.path.join(CSRC, f) for f in ("shard_kernels.hpp", "lamb_kernels.hpp", "probe_kernels.hpp",
                                                  "host_common.hpp")] + [os.path.join(ROOT, "include", "zero_shard.h")]
LIB = os.path.join(PKG, "libzeroshard.so")
ARCH = "gfx950"

HIPCC_FLAGS = [
    "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result",
    "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
]


def hipcc() -> str:
    return os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def build(verbose: bool = False, extra_flags=()) -> str:
    """Compile the library in-tree; returns its path."""
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc(), *HIPCC_FLAGS, *extra_flags, *SOURCES, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


def is_stale() -> bool:
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(d) > t for d in DEPS)


if __name__ == "__main__":
    print(build(verbose=True))
    sys.exit(0)
