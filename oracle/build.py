"""Compile the CPU oracle (test infrastructure) into ``oracle/liboracle.so``.

The flags keep every float operation a single IEEE operation in program
order: no contraction into FMA, no fast-math, no flush-to-zero.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "zpp_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
          "-Wall", "-Wextra", "-Werror"]


def build_oracle(extra_flags=(), out=LIB, src=SRC):
    """Compile the oracle; returns the path of the shared library."""
    tmp = out + ".tmp%d" % os.getpid()
    cmd = ["gcc", *CFLAGS, *extra_flags, src, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build_oracle())
