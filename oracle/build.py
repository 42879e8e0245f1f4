"""Compile the CPU oracle (plain C) into oracle/liboracle.so.

Test infrastructure: only the tests, the smoke check and the benchmark's
CPU-baseline leg load the result.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liboracle.so")


def build(verbose: bool = False, src: str | None = None, out: str | None = None,
          sanitize: bool = False) -> str:
    """Compile `src` (default: the oracle) into `out` (default: oracle/liboracle.so).

    sanitize: AddressSanitizer and UndefinedBehaviorSanitizer build (aborts on
    the first finding); a process loading it needs the gcc ASan runtime
    preloaded (asan_runtime())."""
    src = src or os.path.join(HERE, "deamoe_oracle.c")
    lib = out or LIB
    # -ffp-contract=off: no fused multiply-add, every product and sum rounds
    # separately; no fast-math, so exp and division are the C library's.
    opt = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
           "-fno-sanitize-recover=undefined"] if sanitize else ["-O2"]
    cmd = ["gcc", "-std=gnu11", *opt, "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
           "-fPIC", "-shared", "-Wall", "-Wextra", "-Wno-unused-parameter",
           "-I", HERE, "-o", lib + ".tmp", src, "-lm"]
    if verbose:
        print(" ".join(cmd), file=sys.stderr)
    subprocess.run(cmd, check=True)
    os.replace(lib + ".tmp", lib)
    return lib


def asan_runtime() -> str:
    """Path of gcc's AddressSanitizer runtime (for LD_PRELOAD)."""
    return subprocess.run(["gcc", "-print-file-name=libasan.so"], check=True,
                          capture_output=True, text=True).stdout.strip()


if __name__ == "__main__":
    print(build(verbose=True))
