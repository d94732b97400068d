"""Compile the plain-C oracle into a shared library next to this file.

Test infrastructure only: the product library never links it.  The flags
keep binary32 arithmetic exactly as written (no FMA contraction, no
fast-math, denormals preserved).
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "ifq_oracle.c")
LIB = os.path.join(HERE, "_liboracle.so")

CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
          "-Wall", "-Wextra", "-Werror"]


def build(force: bool = False) -> str:
    """Build _liboracle.so (always when force, else only when missing or stale)."""
    stale = (not os.path.exists(LIB)) or os.path.getmtime(LIB) < os.path.getmtime(SRC)
    if force or stale:
        tmp = LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", *CFLAGS, SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(force="--force" in sys.argv))
