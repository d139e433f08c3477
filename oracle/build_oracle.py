"""Build the CPU oracle shared library (test infrastructure only).

Compiles ``rt3d_oracle.c`` with gcc at -O2 (no fast-math, so float64
arithmetic keeps IEEE semantics) and OpenMP into ``librt3d_oracle.so`` next
to this file.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "rt3d_oracle.c")
LIB = os.path.join(HERE, "librt3d_oracle.so")
CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-Wall", "-Wextra", "-Werror"]
LIBS = ["-lm"]


def build_oracle(force: bool = True) -> str:
    """Compile the oracle; with force=False an existing library is kept."""
    if not force and os.path.exists(LIB):
        return LIB
    tmp = LIB + ".tmp%d" % os.getpid()
    subprocess.run(["gcc", *CFLAGS, SRC, "-o", tmp, *LIBS], check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build_oracle(force=True))
