"""Compile the HIP sources into libsao.so for gfx950 (in-tree, no JIT cache).

Usage: python -m paper_2607_07508_amd.build
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libsao.so")
PROBE_LIB = os.path.join(PKG, "libsao_probe.so")   # bench.py --mfma-ceiling only
ARCH = os.environ.get("SAO_OFFLOAD_ARCH", "gfx950")

SOURCES = ["api.cpp", "runtime.cpp", "head.hip", "scan.hip", "step.hip", "baseline.hip", "loss.hip", "ev.hip", "value.hip"]


def hipcc() -> str:
    for c in (os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc"), shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found (ROCm toolchain required to build libsao.so)")


def _flags():
    return ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
            # packed fp32 VALU ops are kept out of generated code
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-Wno-unused-command-line-argument", "-I", os.path.join(ROOT, "include"), "-I", CSRC]


def _compile(src: str, extra) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc(), *_flags(), *extra, "-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".hip"):
        cmd[1:1] = ["-x", "hip"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {src}\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(extra=(), verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(lambda s: _compile(s, list(extra)), SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    # the measurement probe of bench.py --mfma-ceiling, a library of its own
    pobj = _compile("probe.hip", list(extra))
    ptmp = PROBE_LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", ptmp, pobj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(ptmp, PROBE_LIB)
    if verbose:
        print(f"built {LIB} and {PROBE_LIB}")
    return LIB


# The argument-validation layer alone (api.cpp, which includes no HIP header) with
# host stand-ins for the launchers (host_stub.cpp): a GPU-free library for running
# the host ABI tests under the sanitizers. Never used by the product path.
HOST_CHECK_LIB = os.path.join(BUILD, "libsao_hostcheck.so")


def build_host_check(sanitize: bool = True) -> str:
    os.makedirs(BUILD, exist_ok=True)
    gxx = shutil.which("g++")
    if gxx is None:
        raise RuntimeError("g++ not found")
    san = ["-fsanitize=address,undefined", "-fno-omit-frame-pointer", "-fno-sanitize-recover=undefined"] \
        if sanitize else []
    cmd = [gxx, "-O1", "-g", "-std=c++17", "-fPIC", "-shared", "-Wall", "-Wextra", "-Werror", *san,
           "-I", os.path.join(ROOT, "include"), "-I", CSRC, os.path.join(CSRC, "api.cpp"),
           os.path.join(CSRC, "host_stub.cpp"), "-o", HOST_CHECK_LIB]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"host-check build failed\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return HOST_CHECK_LIB


if __name__ == "__main__":
    build(extra=sys.argv[1:], verbose=True)
