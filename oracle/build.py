"""Build the CPU oracle (test infrastructure only) into oracle/libretopk_oracle.so.

Plain gcc, single-threaded, -O2, ISO C11 (no FMA contraction, no vector
intrinsics, no OpenMP).
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "retopk_oracle.c")
LIB = os.path.join(HERE, "libretopk_oracle.so")


def build(src: str = SRC, out: str = LIB, extra: list[str] | None = None) -> str:
    """Compile `src` into the shared library `out` and return its path."""
    cmd = ["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fPIC", "-shared",
           "-Wall", "-Wextra", "-o", out + ".tmp", src, "-lm"]
    if extra:
        cmd[1:1] = extra
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    print(build(extra=sys.argv[1:] or None))
