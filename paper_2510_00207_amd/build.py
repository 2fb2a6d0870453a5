"""Build libflowmoe.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2510_00207_amd.build [--jobs N]

Every .hip source under csrc/ is compiled to an object and linked into
paper_2510_00207_amd/libflowmoe.so. Always rebuilds.
"""
from __future__ import annotations

import argparse
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
LIB = os.path.join(PKG, "libflowmoe.so")
ARCH = "gfx950"

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
    # code object v5 loads in every HIP runtime this may share a process with
    "-mcode-object-version=5",
    # keep packed-fp32 (v_pk_*_f32) instructions out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{INCLUDE}", f"-I{CSRC}",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libflowmoe)")


def sources() -> list[str]:
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))


def _run(cmd: list[str]) -> None:
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops" not in l and l.strip())
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    if out:
        print(out, file=sys.stderr)


def build(jobs: int | None = None, verbose: bool = True) -> str:
    cc = hipcc()
    os.makedirs(BUILD, exist_ok=True)
    srcs = sources()
    objs = [os.path.join(BUILD, os.path.basename(s)[:-4] + ".o") for s in srcs]
    jobs = jobs or min(8, len(srcs))

    def compile_one(pair):
        src, obj = pair
        _run([cc, *HIPCC_FLAGS, "-c", src, "-o", obj])
        if verbose:
            print(f"[build] compiled {os.path.basename(src)}", flush=True)

    with cf.ThreadPoolExecutor(jobs) as ex:
        list(ex.map(compile_one, zip(srcs, objs)))
    tmp = LIB + ".tmp"
    _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, LIB)
    if verbose:
        print(f"[build] linked {LIB}", flush=True)
    return LIB


# host-side sanitizers for the C ABI front end (argument validation, status
# codes, capacity and workspace arithmetic, the event pool): each -fsanitize
# applies to the host compilation only (-Xarch_host); the device code is built
# as usual
SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host",
            "-fno-omit-frame-pointer"]
SAN_DIR = os.path.join(BUILD, "sanitize")
SAN_LIB = os.path.join(SAN_DIR, "libflowmoe_san.so")


def asan_runtime() -> str:
    """The clang ASan runtime that a process loading the sanitized library
    must preload (its host executable is not instrumented)."""
    llvm = os.path.join(os.path.dirname(os.path.dirname(hipcc())), "llvm", "lib", "clang")
    for ver in sorted(os.listdir(llvm), reverse=True):
        p = os.path.join(llvm, ver, "lib", "linux", "libclang_rt.asan-x86_64.so")
        if os.path.exists(p):
            return p
    raise RuntimeError("clang ASan runtime not found")


def build_sanitized(jobs: int | None = None, verbose: bool = True) -> str:
    """libflowmoe_san.so: abi.hip's host code built with ASan and UBSan, the
    other sources as usual, for host-only tests of the ABI front end."""
    cc = hipcc()
    os.makedirs(SAN_DIR, exist_ok=True)
    srcs = sources()
    objs = [os.path.join(SAN_DIR, os.path.basename(s)[:-4] + ".o") for s in srcs]

    def compile_one(pair):
        src, obj = pair
        extra = SANITIZE if os.path.basename(src) == "abi.hip" else []
        _run([cc, *HIPCC_FLAGS, *extra, "-c", src, "-o", obj])
        if verbose:
            print(f"[build] compiled {os.path.basename(src)}{' (sanitized)' if extra else ''}",
                  flush=True)

    with cf.ThreadPoolExecutor(jobs or min(8, len(srcs))) as ex:
        list(ex.map(compile_one, zip(srcs, objs)))
    _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-Xarch_host",
          "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-Xarch_host",
          "-shared-libasan", "-o", SAN_LIB])
    if verbose:
        print(f"[build] linked {SAN_LIB}", flush=True)
    return SAN_LIB


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=None)
    ap.add_argument("--sanitize", action="store_true",
                    help="build the host-sanitized library for the ABI tests instead")
    a = ap.parse_args()
    if a.sanitize:
        build_sanitized(a.jobs)
    else:
        build(a.jobs)
