"""Build ``liboracle.so`` from ``oracle.c`` with gcc.

Test infrastructure: the oracle is a CPU checker for the GPU library.  It is
built with ``-ffp-contract=off`` so that every multiply and add rounds
separately in fp32, in source order, and with OpenMP for the CPU-baseline
timing (threads never change a result: each output row is computed by one
thread, sequentially).
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
LIB = os.path.join(HERE, "liboracle.so")


def build(verbose: bool = False) -> str:
    cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
           "-fPIC", "-shared", "-Wall", "-Wextra", "-o", LIB + ".tmp", SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
