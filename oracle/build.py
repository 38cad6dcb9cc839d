"""Compile the CPU oracle (test infrastructure) into oracle/libedit_oracle.so.

The oracle is plain C built with the host compiler; it shares no source,
header or flag set with the HIP library of the package.
"""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(HERE, "edit_oracle.c")
LIBRARY = os.path.join(HERE, "libedit_oracle.so")

# -ffp-contract=off: no fused multiply-adds, so every fp64 operation rounds
# exactly as written in the source.
CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math",
          "-Wall", "-Wextra"]


def build_oracle(verbose: bool = False) -> str:
    """Compile the oracle unconditionally; return the library path."""
    tmp = LIBRARY + ".tmp"
    cmd = ["gcc", *CFLAGS, "-o", tmp, SOURCE, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIBRARY)
    return LIBRARY


if __name__ == "__main__":
    print(build_oracle(verbose=True))
