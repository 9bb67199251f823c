"""Build libcmerge.so (the HIP kernels + C ABI) in-tree for gfx950 with hipcc.

Also builds tests/native/libcm_hostcheck.so, a CPU-side harness the tests use
to run the library's BLAKE3 code and the kernels' address maps on the host, and
_build/san/libcmerge_san.so, the same library with its host code built under
AddressSanitizer and UndefinedBehaviorSanitizer for the CPU tests."""

from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libcmerge.so")
HOSTCHECK_SRC = os.path.join(ROOT, "tests", "native", "hostcheck.hip")
HOSTCHECK_LIB = os.path.join(ROOT, "tests", "native", "libcm_hostcheck.so")

ARCH = "gfx950"
SOURCES = ["api.cpp", "hash.hip", "knorm.hip", "order.hip", "paged.hip", "render.hip",
           "render_hash.hip"]
COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
          f"-I{INCLUDE}", f"-I{CSRC}"]
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


# The host side of the C ABI (argument checks, workspace sizing, error
# reporting) built with AddressSanitizer and UndefinedBehaviorSanitizer for the
# CPU tests; device code is not instrumented. The other objects are the normal
# build's. The library leaves the sanitizer runtime's symbols to the process:
# load it with that runtime preloaded (sanitizer_runtime()).
SAN_LIB = os.path.join(BUILD, "san", "libcmerge_san.so")
SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-g"]


def _hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found (ROCm is required to build libcmerge)")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"build step failed: {' '.join(cmd)}\n{out}")
    if verbose and out.strip():
        print(out, flush=True)


def build(verbose: bool = False) -> str:
    hipcc = _hipcc()
    os.makedirs(BUILD, exist_ok=True)
    objs, jobs = [], []
    for src in SOURCES:
        obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
        objs.append(obj)
        lang = ["-x", "hip"] + DEVICE  # hipcc compiles .cpp as HIP too; give it the target
        jobs.append([hipcc, *COMMON, *lang, "-c", os.path.join(CSRC, src), "-o", obj])
    jobs.append([hipcc, *COMMON, "-x", "hip", *DEVICE, "-shared", HOSTCHECK_SRC,
                 "-o", HOSTCHECK_LIB + ".tmp"])
    os.makedirs(os.path.dirname(SAN_LIB), exist_ok=True)
    jobs.append(_san_api_job(hipcc))
    with cf.ThreadPoolExecutor(max_workers=min(len(jobs), os.cpu_count() or 4)) as ex:
        list(ex.map(lambda c: _run(c, verbose), jobs))
    tmp = LIB + ".tmp"
    _run([hipcc, *DEVICE, "-shared", "-fPIC", *objs, "-o", tmp], verbose)
    os.replace(tmp, LIB)
    os.replace(HOSTCHECK_LIB + ".tmp", HOSTCHECK_LIB)
    _link_sanitized(hipcc, verbose)
    return LIB


def sanitizer_runtime() -> str:
    """Path of the compiler's shared AddressSanitizer runtime (it carries the
    UndefinedBehaviorSanitizer handlers as well)."""
    rt = subprocess.run([os.path.join(os.path.dirname(os.path.realpath(_hipcc())), "..", "llvm",
                                      "bin", "clang"), "-print-file-name=libclang_rt.asan-x86_64.so"],
                        capture_output=True, text=True).stdout.strip()
    if not rt or not os.path.exists(rt):
        raise RuntimeError("the compiler's AddressSanitizer runtime was not found")
    return rt


def _san_api_job(hipcc):
    return [hipcc, *COMMON, "-x", "hip", *DEVICE, *SANITIZE, "-c", os.path.join(CSRC, "api.cpp"),
            "-o", os.path.join(os.path.dirname(SAN_LIB), "api.o")]


def _link_sanitized(hipcc, verbose):
    objs = [os.path.join(os.path.dirname(SAN_LIB), "api.o")] + [
        os.path.join(BUILD, os.path.splitext(s)[0] + ".o") for s in SOURCES if s != "api.cpp"]
    tmp = SAN_LIB + ".tmp"
    _run([hipcc, *DEVICE, "-shared", "-fPIC", *objs, "-o", tmp], verbose)
    os.replace(tmp, SAN_LIB)


def build_sanitized(verbose: bool = False) -> str:
    """Rebuild only the sanitized library (the normal objects must exist)."""
    hipcc = _hipcc()
    if not all(os.path.exists(os.path.join(BUILD, os.path.splitext(s)[0] + ".o")) for s in SOURCES):
        build(verbose)
        return SAN_LIB
    os.makedirs(os.path.dirname(SAN_LIB), exist_ok=True)
    _run(_san_api_job(hipcc), verbose)
    _link_sanitized(hipcc, verbose)
    return SAN_LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
