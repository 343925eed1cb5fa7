"""Builds the CPU oracle (test infrastructure) into oracle/liblsgd_oracle.so.

gcc, -O2, no -march (so no FMA instructions exist to contract into), explicit
-ffp-contract=off and no fast-math: every C operation is one IEEE binary32 or
binary64 operation rounded to nearest-even, with subnormals kept.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liblsgd_oracle.so")


def build(verbose: bool = False) -> str:
    src = os.path.join(HERE, "lsgd_oracle.c")
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math",
           "-fexcess-precision=standard", "-Wall", "-Wextra", "-Werror",
           "-shared", "-fPIC", "-o", tmp, src]
    if verbose:
        print(" ".join(cmd), file=sys.stderr)
    subprocess.run(cmd, check=True, cwd=HERE)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
