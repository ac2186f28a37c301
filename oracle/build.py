"""Compile the CPU oracle (oracle.c) into oracle/liboracle.so with gcc."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liboracle.so")


# Host sanitizers for a checking build of the oracle (gcc, CPU only):
# out-of-bounds and use-after-free accesses, and undefined behaviour such as
# signed overflow or misaligned loads, each stopping the process.
SANITIZE_FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                  "-fno-omit-frame-pointer", "-g"]


def build(verbose: bool = False, sanitize: bool = False, out: str | None = None,
          src: str | None = None) -> str:
    """Compiles oracle.c (or `src`, a copy of it) into `out` (default:
    liboracle.so beside it); with sanitize=True an instrumented build for the
    sanitizer test."""
    src = src or os.path.join(HERE, "oracle.c")
    out = out or LIB
    tmp = out + ".tmp"
    cmd = ["gcc", "-std=c11", "-O1" if sanitize else "-O2", "-ffp-contract=off", "-fno-fast-math",
           "-fPIC", "-shared", "-Wall", "-Wextra", "-I", HERE] + (SANITIZE_FLAGS if sanitize else []) + \
          ["-o", tmp, src, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
