"""Compile the fp64 CPU oracle (oracle.c: triangle attention; ln_linear.c:
fused layer-norm + linear projection) into liboracle.so with gcc.

Test infrastructure: only the tests, the smoke check and the benchmark's
CPU-baseline leg load the result.  build() makes generic x86-64 code (no
-march=native), so the library built here also runs on another host;
build_native() makes an -O3 -march=native copy for the host it runs on, which
the benchmark times.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
SRC_LNL = os.path.join(HERE, "ln_linear.c")
LIB = os.path.join(HERE, "liboracle.so")


NATIVE_LIB = os.path.join(HERE, "liboracle_native.so")
NATIVE_FLAGS = ["-O3", "-march=native", "-fopenmp"]


def build_native(verbose: bool = False) -> str:
    """The same sources built for the host this runs on (-O3 -march=native):
    what the benchmark's CPU-baseline leg times.  Not used by the tests."""
    cmd = ["gcc", *NATIVE_FLAGS, "-fPIC", "-shared", "-std=c11", "-Wall",
           SRC, SRC_LNL, "-o", NATIVE_LIB + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(NATIVE_LIB + ".tmp", NATIVE_LIB)
    return NATIVE_LIB


def build(verbose: bool = False) -> str:
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall",
           SRC, SRC_LNL, "-o", LIB + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
