"""Build the oracle's C solvers into oracle/_liboracle.so (test infrastructure).

Plain C compiled with gcc for the host; nothing here touches the GPU path.
Run as `python -m oracle.build` or call build()."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "_liboracle.so")
SOURCES = [os.path.join(HERE, "csrc", f) for f in ("hungarian.c", "ssp.c")]


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-shared", "-fPIC", "-o", tmp, *SOURCES, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


def ensure_built() -> str:
    """Build only when the library is missing or older than a source."""
    if os.path.exists(LIB):
        mtime = os.path.getmtime(LIB)
        if all(os.path.getmtime(s) <= mtime for s in SOURCES):
            return LIB
    return build()


if __name__ == "__main__":
    print(build(verbose=True))
