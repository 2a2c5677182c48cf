"""Compile the CPU oracle (plain C++, g++) into ``oracle/liboracle.so``.

Test infrastructure: see the package docstring.
"""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "scn_oracle.cpp")
LIB_PATH = os.environ.get("SCN_ORACLE_LIB") or os.path.join(HERE, "liboracle.so")


def build(verbose: bool = False) -> str:
    tmp = LIB_PATH + ".tmp%d" % os.getpid()
    cmd = ["g++", "-O2", "-std=c++17", "-shared", "-fPIC", "-Wall", SRC, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose=True))
