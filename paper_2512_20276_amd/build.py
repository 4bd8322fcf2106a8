"""Builds libactionflow.so (HIP kernels for gfx950 + the C ABI) in the package directory."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
OUT = os.path.join(PKG, "libactionflow.so")
BUILD_DIR = os.path.join(PKG, "_build")

HIP_SOURCES = ["af_gemm.hip", "af_attention.hip", "af_kernels.hip", "af_noalloc.hip"]
HOST_SOURCES = ["af_ring.cpp", "af_model.cpp"]

# Packed-fp32 instructions are disabled for all device code (hipcc makes them from plain float
# code otherwise); the host pass warns that it does not know the feature, which is harmless.
DEVICE_FLAGS = ["--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON = ["-O3", "-fPIC", "-std=c++17", "-Wall", "-Wno-unused-function", f"-I{ROOT}/include"]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found (ROCm is required to build the HIP library)")


def _run(cmd):
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in p.stdout.splitlines() if "packed-fp32-ops" not in l)
    if p.returncode != 0:
        raise RuntimeError(f"build step failed ({p.returncode}): {' '.join(cmd)}\n{out}")
    return out


HEADERS = [os.path.join(CSRC, "af_internal.h"), os.path.join(CSRC, "af_device.h"),
           os.path.join(ROOT, "include", "actionflow.h")]


def _stale(src: str, obj: str) -> bool:
    if not os.path.exists(obj):
        return True
    t = os.path.getmtime(obj)
    return any(os.path.getmtime(p) > t for p in [src, *HEADERS])


def build(verbose: bool = False, changed_only: bool = False) -> str:
    """Compile every source (with changed_only: those newer than their object or than a header)
    and link the shared library; returns its path."""
    cc = hipcc()
    os.makedirs(BUILD_DIR, exist_ok=True)
    jobs, objs = [], []
    for srcs, flags in ((HIP_SOURCES, DEVICE_FLAGS), (HOST_SOURCES, [])):
        for src in srcs:
            path, obj = os.path.join(CSRC, src), os.path.join(BUILD_DIR, src + ".o")
            objs.append(obj)
            if not changed_only or _stale(path, obj):
                jobs.append([cc, *COMMON, *flags, "-c", path, "-o", obj])
    logs = []
    if jobs:
        with ThreadPoolExecutor(max_workers=len(jobs)) as ex:
            logs = list(ex.map(_run, jobs))
    tmp = OUT + ".tmp"
    logs.append(_run([cc, "-shared", "-fPIC", *DEVICE_FLAGS, *objs, "-o", tmp]))
    os.replace(tmp, OUT)
    if verbose:
        for l in logs:
            if l.strip():
                print(l)
    return OUT


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, changed_only="--changed" in sys.argv))
