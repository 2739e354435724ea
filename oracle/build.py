"""Compile the fp64 attention oracle (plain C, gcc) into oracle/liboracle_attn.so.

Test infrastructure: the library this builds is loaded only by the test suite,
the smoke check and the bench's CPU-baseline leg.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "attn_oracle.c")
LIB = os.path.join(HERE, "liboracle_attn.so")


def build(src: str = SRC, out: str = LIB, extra=()) -> str:
    """Build ``src`` into the shared library ``out`` and return its path.

    -O2 without -ffast-math: the oracle keeps IEEE double semantics and its
    written summation order."""
    tmp = out + ".tmp"
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-Werror", "-fPIC", "-shared",
           *extra, "-o", tmp, src, "-lm", "-lpthread"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(*sys.argv[1:2]))
