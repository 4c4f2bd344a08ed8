"""Builds the oracle's C library (test infrastructure; see ``oracle/__init__``).

``python -m oracle.build`` or ``oracle.build.build()``; host gcc with OpenMP.
"""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "gdn_oracle.c")
LIB_PATH = os.path.join(HERE, "libgdn_oracle.so")


def build(verbose: bool = False) -> str:
    """Compiles ``gdn_oracle.c`` into ``libgdn_oracle.so`` next to it."""
    tmp = LIB_PATH + ".tmp"
    cmd = ["gcc", "-O2", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
           "-std=c11", "-Wall", "-Wextra", "-o", tmp, SRC, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose=True))
