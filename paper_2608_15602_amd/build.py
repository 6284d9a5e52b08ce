"""Build libfluxbin.so (HIP for gfx950) in-tree with hipcc.

Usage: python -m paper_2608_15602_amd.build [--jobs N] [--host-sanitizers]
The shared library lands next to this file, where the Python binding loads it from. --host-sanitizers also builds
libfluxbin_hostsan.so: the same library with its host code (fluxbin_host.cpp: validation, sizes, launch planning,
headers) instrumented by AddressSanitizer and UndefinedBehaviorSanitizer, for CPU-only tests (the device code is the
ordinary build's; no sanitizer touches GPU code).
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJDIR = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libfluxbin.so")
SAN_LIB = os.path.join(HERE, "libfluxbin_hostsan.so")
# host-only sanitizers: each -fsanitize applies to the host compilation (-Xarch_host), never to GPU code
SAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-Xarch_host",
             "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]

SOURCES = ["fluxbin_host.cpp", "fluxbin_pack.hip", "fluxbin_gemv.hip", "fluxbin_gemm_batch.hip",
           "fluxbin_gemm_mfma.hip", "fluxbin_rc.hip", "fluxbin_noalloc.hip",
           "fluxbin_gemv_rows.hip", "fluxbin_gemm_mfma_rows.hip"]
ARCH = "gfx950"

# Packed-FP32 instructions are kept out of the generated code (plain float code only).
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Wall", "-Wno-unused-function",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-I", INCLUDE, "-I", CSRC]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _compile(src: str) -> str:
    obj = os.path.join(OBJDIR, os.path.basename(src) + ".o")
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    cmd = [hipcc()] + COMMON + lang + ["-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    warn = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l and l.strip())
    if warn:
        sys.stderr.write(warn + "\n")
    return obj


def build(jobs: int = 4, verbose: bool = True) -> str:
    os.makedirs(OBJDIR, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=max(1, jobs)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


def asan_runtime() -> str:
    """Path of the compiler's shared AddressSanitizer runtime (a Python process loading the sanitized library needs it
    preloaded)."""
    clang = os.path.join(os.path.dirname(os.path.dirname(os.path.realpath(hipcc()))), "llvm", "bin", "clang++")
    r = subprocess.run([clang, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True)
    return r.stdout.strip()


def build_host_sanitized(verbose: bool = True) -> str:
    """libfluxbin_hostsan.so: fluxbin_host.cpp compiled with host ASan + UBSan, linked with the device objects of the
    ordinary build (built first if missing)."""
    os.makedirs(OBJDIR, exist_ok=True)
    objs = []
    for src in SOURCES:
        obj = os.path.join(OBJDIR, os.path.basename(src) + ".o")
        if src == "fluxbin_host.cpp":
            obj = os.path.join(OBJDIR, "fluxbin_host_san.o")
            cmd = [hipcc()] + COMMON + SAN_FLAGS + ["-c", os.path.join(CSRC, src), "-o", obj]
            r = subprocess.run(cmd, capture_output=True, text=True)
            if r.returncode != 0:
                raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
        elif not os.path.exists(obj):
            obj = _compile(src)
        objs.append(obj)
    tmp = SAN_LIB + ".tmp"
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", "-shared-libsan"] + SAN_FLAGS[:4] + ["-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, SAN_LIB)
    if verbose:
        print(f"built {SAN_LIB}")
    return SAN_LIB


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=3)
    ap.add_argument("--host-sanitizers", action="store_true")
    args = ap.parse_args()
    build(args.jobs)
    if args.host_sanitizers:
        build_host_sanitized()
