"""Test infrastructure only: compiles the CPU oracle (conv2d_oracle.c) with gcc.

The oracle is a plain host library; it shares no source, header or build step
with the HIP library of the package.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "conv2d_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")


def build(force=True):
    """Compile liboracle.so next to its source (no -ffast-math: the oracle's
    fp64 sums must keep their written order)."""
    if not force and os.path.exists(LIB) and os.path.getmtime(LIB) >= os.path.getmtime(SRC):
        return LIB
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-fno-fast-math",
           "-Wall", "-Wextra", SRC, "-o", tmp]
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
