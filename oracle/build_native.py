"""Build the oracle's C part (oracle/libblake3_ref.so) with gcc.

Test infrastructure: the CPU oracle's BLAKE3 lives in blake3_ref.c and is
loaded by cmerge_oracle through ctypes. Nothing in the product path builds on
it; __graft_entry__.build() compiles it beside the library so that the tests,
smoke() and the benchmark's CPU baseline find it."""

from __future__ import annotations

import os
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "blake3_ref.c")
LIB = os.path.join(HERE, "libblake3_ref.so")


def build(verbose: bool = False) -> str:
    cc = os.environ.get("CC") or shutil.which("gcc") or shutil.which("cc")
    if not cc:
        raise RuntimeError("no C compiler found for the oracle (gcc)")
    tmp = LIB + ".tmp"
    cmd = [cc, "-O2", "-std=c99", "-Wall", "-Wextra", "-shared", "-fPIC", SRC, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"oracle build failed: {' '.join(cmd)}\n{r.stdout}{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
