"""Build libosprey.so (HIP for gfx950) in-tree.

    python -m paper_2609_09338_amd.build [--jobs N] [--debug]

Every source is compiled with hipcc into _build/, then linked into
paper_2609_09338_amd/libosprey.so.  Always recompiles (it is the build check).
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
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libosprey.so")
SOURCES = ["gemv.hip", "gemv_taps.hip", "gemv_qkv.hip", "gemv_resid.hip", "gemv_swiglu.hip",
           "gemv_logits.hip", "gemm_mfma.hip", "skinny.hip", "rows.hip", "attention.hip", "sample.hip", "verify.hip", "verify_static.hip",
           "state.hip", "tree.hip", "osprey.cpp"]
ARCH = "gfx950"


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found (ROCm is required to build libosprey)")


def flags(debug: bool):
    f = [f"--offload-arch={ARCH}", "-std=c++17", "-fPIC", "-fvisibility=hidden",
         # packed fp32 instructions stay off (correctness of some forms on this hardware)
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-Wno-unused-result"]
    f += ["-O0", "-g"] if debug else ["-O3"]
    return f


def compile_one(src: str, debug: bool) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc()] + flags(debug) + ["-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".cpp"):
        cmd[1:1] = ["-x", "hip"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compiling {src} failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(jobs: int = 6, debug: bool = False, verbose: bool = True) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=max(1, jobs)) as ex:
        objs = list(ex.map(lambda s: compile_one(s, debug), SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"linking failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}", file=sys.stderr)
    return LIB


# Sources whose host code holds the library's logic (validation, planning, the slot
# state machine, the graph and no-allocation entry points); the other sources' host
# code is kernel-launch stubs.
HOST_LOGIC = ["osprey.cpp", "verify_static.hip"]
SANITIZED = os.path.join(BUILD, "sanitized", "libosprey.so")


def build_sanitized(verbose: bool = True) -> str:
    """A build of the library whose host code in HOST_LOGIC is instrumented with
    AddressSanitizer and UndefinedBehaviorSanitizer (host only: no GPU code is
    instrumented; the other objects are the regular ones).  The sanitizer runtime is
    not linked in: load the library into a process that preloads it."""
    if not all(os.path.exists(os.path.join(BUILD, os.path.splitext(s)[0] + ".o")) for s in SOURCES):
        build(verbose=False)
    out = os.path.dirname(SANITIZED)
    os.makedirs(out, exist_ok=True)
    objs = []
    for src in SOURCES:
        obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
        if src in HOST_LOGIC:
            obj = os.path.join(out, os.path.splitext(src)[0] + ".o")
            cmd = [hipcc()] + flags(False) + [
                "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer",
                "-g", "-c", os.path.join(CSRC, src), "-o", obj]
            if src.endswith(".cpp"):
                cmd[1:1] = ["-x", "hip"]
            r = subprocess.run(cmd, capture_output=True, text=True)
            if r.returncode != 0:
                raise RuntimeError(f"compiling {src} (sanitized) failed:\n{r.stdout}\n{r.stderr}")
        objs.append(obj)
    tmp = SANITIZED + ".tmp"
    r = subprocess.run([hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs,
                       capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"linking the sanitized library failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, SANITIZED)
    if verbose:
        print(f"built {SANITIZED}", file=sys.stderr)
    return SANITIZED


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=6)
    ap.add_argument("--debug", action="store_true")
    ap.add_argument("--sanitize", action="store_true",
                    help="build the host-sanitized library instead (see build_sanitized)")
    args = ap.parse_args()
    if args.sanitize:
        build_sanitized()
    else:
        build(args.jobs, args.debug)
