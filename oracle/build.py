"""Compile the plain-C oracle into ``oracle/liboracle.so`` with gcc.

Test infrastructure only: the product library never links or loads it.
Flags keep every float addition a single IEEE binary32 add (no contraction,
no fast-math, SSE arithmetic on x86-64).
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "nuna_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

CFLAGS = ["-O1", "-std=c99", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math",
          "-fexcess-precision=standard", "-Wall", "-Wextra"]


def build(out=LIB, extra_flags=()):
    """Build the oracle library; ``extra_flags`` lets tests build variants."""
    tmp = out + ".tmp"
    cmd = ["gcc", *CFLAGS, *extra_flags, SRC, "-o", tmp]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build())
