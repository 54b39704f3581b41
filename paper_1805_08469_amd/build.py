"""Build libgem.so (HIP kernels + C ABI) for gfx950 with hipcc, in-tree.

Floating-point flags are part of the numerics: no contraction
(-ffp-contract=off), IEEE division and square root (hipcc's default),
denormals kept (no flush flag), and no packed-FP32 instructions.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libgem.so")
SOURCES = [os.path.join(CSRC, f) for f in ("gem_kernels.hip", "gem_api.cpp")]
# Device self-tests of the numerics (used by the test suite only).
SELFTEST_LIB = os.path.join(HERE, "libgem_selftest.so")
SELFTEST_SOURCES = [os.path.join(CSRC, "gem_selftest.hip")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off", "-fno-fast-math",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
]


def _link(out: str, sources, verbose: bool, extra) -> None:
    cmd = [HIPCC, *FLAGS, *extra, "-o", out + ".tmp", *sources]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)


def build(verbose: bool = False, extra=()) -> str:
    _link(LIB, SOURCES, verbose, extra)
    _link(SELFTEST_LIB, SELFTEST_SOURCES, verbose, extra)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
