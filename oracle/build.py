"""Build the oracle's shared library (test infrastructure, plain C, fp64).

gcc -O2 -ffp-contract=off keeps every a*b+c as two IEEE roundings unless the
source writes fma() explicitly; OpenMP runs independent KV heads in parallel.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "certkv_oracle.c")
LIB = os.path.join(HERE, "libcertkv_oracle.so")


def build(verbose: bool = False) -> str:
    cmd = ["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
           "-std=c99", "-fPIC", "-shared", "-Wall", "-o", LIB + ".tmp", SRC, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
