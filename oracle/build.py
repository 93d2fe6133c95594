"""Build step for the CPU oracle (test infrastructure only).

Compiles ``oracle.c`` with gcc into ``liboracle.so`` beside it.  Plain
``-O2``, no fast-math, so every fp64 operation is the IEEE operation the
source spells out.  OpenMP only splits the independent per-element loop.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
LIB = os.path.join(HERE, "liboracle.so")


def build(verbose: bool = False, src: str = SRC, out: str = LIB) -> str:
    tmp = out + ".tmp"
    cmd = [
        "gcc", "-std=c11", "-O2", "-fno-fast-math", "-ffp-contract=off",
        "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra",
        "-I", HERE, "-o", tmp, src, "-lm",
    ]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
