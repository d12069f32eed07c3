"""Build the CPU oracle shared library (test infrastructure only).

Compiles ``oracle.c`` into ``liboracle.so`` beside it with gcc, IEEE
binary32 semantics (no fast-math) and OpenMP.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liboracle.so")


def build(verbose: bool = False) -> str:
    cmd = [
        "gcc", "-O2", "-fno-fast-math", "-std=c11", "-fopenmp", "-shared",
        "-fPIC", "-Wall", "-Wextra", "-o", LIB + ".tmp",
        os.path.join(HERE, "oracle.c"), "-lm",
    ]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
