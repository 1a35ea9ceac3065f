"""Builds the fp64 CPU oracle (oracle/liblppref.so) with gcc.

Test infrastructure: the oracle checks the HIP library and is never part of
its product path.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "lppref.c")
LIB = os.path.join(HERE, "liblppref.so")


def build(force: bool = True) -> str:
    if not force and os.path.exists(LIB) and os.path.getmtime(LIB) >= os.path.getmtime(SRC):
        return LIB
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall", "-Wno-unknown-pragmas",
           "-o", tmp, SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


def build_native(out_dir: str) -> str:
    """A copy of the oracle compiled for the host it runs on (-O3
    -march=native), for timing it as the CPU baseline; the tests use the
    portable build above."""
    os.makedirs(out_dir, exist_ok=True)
    out = os.path.join(out_dir, "liblppref_native.so")
    cmd = ["gcc", "-O3", "-march=native", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall", "-Wno-unknown-pragmas",
           "-o", out, SRC, "-lm"]
    subprocess.run(cmd, check=True)
    return out


if __name__ == "__main__":
    print(build(force="--if-stale" not in sys.argv))
