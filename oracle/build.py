"""Compile the oracle (test infrastructure) into oracle/liboracle.so with gcc.

Flags: -O2 -ffp-contract=off, no -ffast-math, so every float operation in
fc_oracle.c is one IEEE-754 binary32 operation rounded to nearest even.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "fc_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")
CFLAGS = ["-O2", "-ffp-contract=off", "-fno-fast-math", "-std=c11", "-fPIC", "-shared",
          "-Wall", "-Wextra"]


def build(src=SRC, lib=LIB, extra=()):
    cmd = ["gcc", *CFLAGS, *extra, src, "-o", lib + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(lib + ".tmp", lib)
    return lib


if __name__ == "__main__":
    print(build(extra=sys.argv[1:]))
