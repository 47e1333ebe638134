"""Build the CPU oracle (liboracle.so) with gcc.

-ffp-contract=off and no fast-math: every binary32 operation in the oracle
is one correctly rounded IEEE-754 operation in the written order.  The
optional `defines` and `src` arguments let a test build a copy of the oracle
with a planted mistake into another directory.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liboracle.so")

CFLAGS = ["-std=c11", "-O2", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math",
          "-Wall", "-Wextra"]


def build(out=LIB, src=None, include_dir=HERE):
    src = src or os.path.join(HERE, "oracle.c")
    subprocess.run(["gcc"] + CFLAGS + ["-I", include_dir, "-o", out, src, "-lm"], check=True)
    return out


if __name__ == "__main__":
    build()
