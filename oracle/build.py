"""Compile the CPU oracle (plain C) into ``oracle/libtlc_ref.so``.

Test infrastructure only: the library is loaded by the test suite, the smoke
check and the benchmark's CPU-baseline leg, never by the product path.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libtlc_ref.so")

# No fast-math and no contraction: fp32 division and rintf must be the IEEE
# operations the paper's equations name.
CFLAGS = ["-std=c11", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fPIC",
          "-shared", "-Wall", "-Wextra", "-Werror"]


def build(verbose=False):
    src = os.path.join(HERE, "tlc_ref.c")
    tmp = LIB + ".tmp"
    cmd = ["gcc", *CFLAGS, "-o", tmp, src, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
