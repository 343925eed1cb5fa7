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


CFLAGS = ["-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fexcess-precision=standard",
          "-Wall", "-Wextra", "-Werror"]


def build(verbose: bool = False, src_dir: str = HERE, out: str = LIB, cflags=None) -> str:
    """Compile lsgd_oracle.c from `src_dir` into `out` (defaults: this
    directory's source and library)."""
    src = os.path.join(src_dir, "lsgd_oracle.c")
    tmp = out + ".tmp%d" % os.getpid()
    cmd = ["gcc"] + (cflags if cflags is not None else CFLAGS) + ["-shared", "-fPIC", "-o", tmp, src, "-lm"]
    if verbose:
        print(" ".join(cmd), file=sys.stderr)
    subprocess.run(cmd, check=True, cwd=src_dir)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
