"""Build the CPU oracle shared library (test infrastructure only).

Compiles ``oracle.c`` into ``liboracle.so`` beside it with gcc, IEEE
binary32 semantics (no fast-math) and OpenMP.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liboracle.so")


def compile_source(c_path: str, out_path: str, verbose: bool = False) -> str:
    """Compile one C source with the oracle's flags into a shared library."""
    cmd = [
        "gcc", "-O2", "-fno-fast-math", "-std=c11", "-fopenmp", "-shared",
        "-fPIC", "-Wall", "-Wextra", "-I", HERE, "-o", out_path + ".tmp", c_path, "-lm",
    ]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(out_path + ".tmp", out_path)
    return out_path


def build(verbose: bool = False) -> str:
    return compile_source(os.path.join(HERE, "oracle.c"), LIB, verbose)


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
