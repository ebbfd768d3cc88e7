"""Builds libpace.so (the HIP library behind include/pace.h) for gfx950 with hipcc.

Usage: python -m paper_2608_27206_amd.build [--jobs N]
Every call recompiles all sources (the build check must compile each time).
"""
from __future__ import annotations

import argparse
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libpace.so")
BUILD = os.path.join(HERE, "_build")
SOURCES = ["abi.cpp", "apc.hip", "attention.hip", "ddae.hip", "preview.hip"]
ARCH = "gfx950"
# Packed-FP32 instructions are switched off for all device code.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
           "-Wno-unused-function", "-I", os.path.join(ROOT, "include"), "-c",
           os.path.join(CSRC, src), "-o", obj] + DEVICE_FLAGS
    if src.endswith(".cpp"):
        cmd = [hipcc(), "-O3", "-std=c++17", "-fPIC", "-Wall", "-D__HIP_PLATFORM_AMD__",
               "-I", os.path.join(ROOT, "include"), "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    errs = "\n".join(l for l in (r.stderr or "").splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {src}\n{errs}")
    return obj


# Host-side AddressSanitizer + UndefinedBehaviorSanitizer build of the whole library (device code is
# compiled exactly as in the normal build: every -fsanitize= applies to the host pass only).  It
# checks the C ABI's argument handling, host metadata checks and launch set-up; load it with the
# clang sanitizer runtime preloaded (tests/test_abi_sanitized.py does).
SANITIZED_OUT = os.path.join(BUILD, "sanitized", "libpace_sanitized.so")
SANITIZE_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                  "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]


def sanitizer_runtime() -> str:
    """The clang ASan runtime (it carries the UBSan handlers) that a sanitized library needs."""
    import glob
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not hits:
        raise RuntimeError("clang ASan runtime not found under /opt/rocm/llvm")
    return hits[-1]


def _compile_sanitized(src: str) -> str:
    out_dir = os.path.dirname(SANITIZED_OUT)
    obj = os.path.join(out_dir, os.path.splitext(src)[0] + ".o")
    inc = ["-I", os.path.join(ROOT, "include")]
    if src.endswith(".cpp"):
        cmd = [hipcc(), "-O1", "-g", "-std=c++17", "-fPIC", "-D__HIP_PLATFORM_AMD__"] + SANITIZE_FLAGS + inc
    else:
        cmd = [hipcc(), f"--offload-arch={ARCH}", "-O3", "-g", "-std=c++17", "-fPIC"] + SANITIZE_FLAGS + inc + \
              DEVICE_FLAGS
    cmd += ["-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        errs = "\n".join(l for l in (r.stderr or "").splitlines() if "packed-fp32-ops" not in l)
        raise RuntimeError(f"sanitized compile failed: {src}\n{errs}")
    return obj


def build_sanitized(jobs: int = 4, verbose: bool = True) -> str:
    os.makedirs(os.path.dirname(SANITIZED_OUT), exist_ok=True)
    with ThreadPoolExecutor(max_workers=max(1, jobs)) as ex:
        objs = list(ex.map(_compile_sanitized, SOURCES))
    tmp = SANITIZED_OUT + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-shared-libsan"] + SANITIZE_FLAGS + \
          ["-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"sanitized link failed\n{r.stderr}")
    os.replace(tmp, SANITIZED_OUT)
    if verbose:
        print(f"built {SANITIZED_OUT}")
    return SANITIZED_OUT


def build(jobs: int = 4, verbose: bool = True) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=max(1, jobs)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = OUT + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed\n{r.stderr}")
    os.replace(tmp, OUT)
    if verbose:
        print(f"built {OUT}")
    return OUT


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=4)
    ap.add_argument("--sanitized", action="store_true",
                    help="also build the host-sanitized (ASan + UBSan) library for the C ABI tests")
    a = ap.parse_args()
    build(a.jobs)
    if a.sanitized:
        build_sanitized(a.jobs)
    sys.exit(0)
