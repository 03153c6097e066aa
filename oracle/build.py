"""Compile the CPU oracle (``lmoracle.c``) into ``liblmoracle.so`` with gcc.

Test infrastructure only; see ``oracle/__init__.py``.
"""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "lmoracle.c")
LIB_PATH = os.path.join(HERE, "liblmoracle.so")


def build() -> str:
    """Compile the oracle. -O2 without -ffast-math keeps IEEE fp64 semantics
    (no reassociation, no contraction into fma)."""
    tmp = LIB_PATH + f".tmp{os.getpid()}"
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
           "-Wall", "-Wextra", "-o", tmp, SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    print(build())
