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
# AddressSanitizer + UndefinedBehaviorSanitizer build of the same source, for
# running the pin suites against it (ORACLE_LIB=<this path>, with gcc's ASan
# runtime preloaded into the Python process).
LIB_ASAN = os.path.join(HERE, "liboracle_asan.so")


def build(verbose: bool = False, sanitize: bool = False) -> str:
    out = LIB_ASAN if sanitize else LIB
    extra = ["-fsanitize=address,undefined", "-fno-omit-frame-pointer", "-fno-sanitize-recover=undefined",
             "-g"] if sanitize else []
    cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
           "-fPIC", "-shared", "-Wall", "-Wextra", *extra, "-o", out + ".tmp", SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    import sys
    print(build(verbose=True, sanitize="--sanitize" in sys.argv))
