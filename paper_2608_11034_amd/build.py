"""Builds libc3.so, the gfx950 HIP library behind include/c3.h, and
libc3_oob.so, the host-only hang-localization library behind
include/c3_oob.h (g++, no HIP: observer processes never touch a GPU).

hipcc compiles every source of csrc/ for gfx950 only:
  -O3, no floating-point contraction (the statistical vote and the AdamW
  replay must round like their plain definitions; sums use explicit fma),
  correctly rounded fp32 division and square root, fp32/fp16 denormals
  kept, packed-fp32 instructions disabled.
"""
import glob
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libc3.so")
OOB_LIB = os.path.join(HERE, "libc3_oob.so")
OOB_SRC = os.path.join(CSRC, "oob", "c3_oob.cpp")
OOB_BENCH = os.path.join(HERE, "c3_oob_bench")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CXX = os.environ.get("CXX", "g++")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off", "-fno-gpu-flush-denormals-to-zero",
    "-fhip-fp32-correctly-rounded-divide-sqrt",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.cpp")))


def build_oob(verbose: bool = False) -> str:
    cmd = [CXX, "-std=c++17", "-O2", "-fPIC", "-shared", "-Wall", "-Wextra", OOB_SRC,
           "-o", OOB_LIB + ".tmp", "-lrt"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(OOB_LIB + ".tmp", OOB_LIB)
    cmd = [CXX, "-std=c++17", "-O2", "-Wall", "-Wextra", "-pthread",
           os.path.join(CSRC, "oob", "c3_oob_bench.cpp"), OOB_SRC, "-o", OOB_BENCH + ".tmp", "-lrt"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(OOB_BENCH + ".tmp", OOB_BENCH)
    return OOB_LIB


def build(verbose: bool = False, extra=None) -> str:
    cmd = [HIPCC] + FLAGS + (extra or []) + ["-I", os.path.join(HERE, "..", "include")] + \
        sources() + ["-o", LIB + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    build_oob(verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
