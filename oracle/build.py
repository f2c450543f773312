"""Build the CPU oracle (test infrastructure only) into oracle/liboracle.so.

Plain gcc, fp64, OpenMP over independent outputs; no fast-math, so every
result is the arithmetic the C source spells out."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "quan_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")


def build(src: str = SRC, lib: str = LIB, verbose: bool = False) -> str:
    cmd = ["gcc", "-std=c99", "-O2", "-fopenmp", "-fPIC", "-shared",
           "-Wall", "-Wextra", "-Werror", "-o", lib + ".tmp", src, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(lib + ".tmp", lib)
    return lib


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
