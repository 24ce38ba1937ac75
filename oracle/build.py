"""Compile the CPU oracle (test infrastructure) into oracle/liborloj_oracle.so."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "orloj_oracle.c")
LIB = os.path.join(HERE, "liborloj_oracle.so")


def compile_oracle(src: str = SRC, out: str = LIB, extra=()) -> str:
    """Build a shared object from ``src``; strict IEEE fp64 (no fast-math,
    no FMA contraction)."""
    tmp = out + ".tmp"
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-fPIC", "-shared",
           "-ffp-contract=off", *extra, src, "-lm", "-o", tmp]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def build() -> str:
    return compile_oracle()


if __name__ == "__main__":
    print(build(), file=sys.stderr)
