"""Build oracle/liboracle.so, the plain C oracle (test infrastructure), with gcc.

    python oracle/build.py

IEEE binary32 arithmetic as written (no fast-math, no contraction); OpenMP spreads
the elements of each chunk (and of each tensor copy) over threads.
"""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liboracle.so")
SRC = os.path.join(HERE, "csrc", "oracle.c")
FLAGS = ["-O2", "-std=c11", "-fno-fast-math", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared", "-Wall",
         "-Wextra", "-Werror"]


def build() -> str:
    tmp = LIB + f".tmp{os.getpid()}"
    subprocess.run(["gcc", *FLAGS, "-o", tmp, SRC], check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
