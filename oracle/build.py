"""Build the oracle's C library with gcc (test infrastructure).

    python oracle/build.py

The library is portable x86-64 code (no -march=native) so that a copy built in
one container runs on another host. The SHA-256 of the source it was built from
is compiled into it, so a stale library is recognised by content, not by file
times. Building starts a compiler process: do it before the GPU is initialised
(the build entry point and the test configuration hook do), never from a
process that has touched the GPU.
"""
from __future__ import annotations

import hashlib
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "pcr_oracle.c")
LIB = os.path.join(HERE, "libpcr_oracle.so")


def source_sha256() -> str:
    with open(SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall", "-Wextra",
           f'-DPCR_ORACLE_SOURCE_SHA256="{source_sha256()}"', SRC, "-o", tmp, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


def is_current() -> bool:
    """True if the library exists and was built from the current source."""
    if not os.path.exists(LIB):
        return False
    with open(LIB, "rb") as f:
        return source_sha256().encode() in f.read()


def ensure_built() -> str:
    """Build only if no library exists or it was built from another source. Call it
    only before the GPU is initialised (it may start the compiler)."""
    if not is_current():
        build()
    return LIB


def require_built() -> str:
    """The library's path; raises if it is missing or stale (never compiles)."""
    if not is_current():
        raise RuntimeError(f"{LIB} is missing or was built from another source than {SRC}: build it "
                           "before the GPU is initialised (python oracle/build.py, or __graft_entry__.build())")
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
    sys.exit(0)
