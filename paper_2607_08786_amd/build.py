"""Builds libusp.so (host encoder, C ABI and gfx950 kernels) in-tree with hipcc."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libusp.so")
SOURCES = ["usp_abi.cpp", "usp_encode.cpp", "usp_kernels.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Packed fp32 VALU forms are disabled for all device code.
DEVICE_FLAGS = ["--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def build(verbose: bool = False) -> str:
    srcs = [os.path.join(CSRC, s) for s in SOURCES]
    tmp = LIB + ".tmp"
    cmd = [HIPCC, *DEVICE_FLAGS, "-O3", "-std=c++17", "-fPIC", "-shared", "-Wall",
           "-Wno-unused-result", "-I", os.path.join(ROOT, "include"), *srcs, "-o", tmp, "-lpthread"]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed building libusp.so")
    os.replace(tmp, LIB)
    build_probe(verbose)
    build_dense_ref(verbose)
    return LIB


PROBE_LIB = os.path.join(HERE, "libusp_probe.so")


def build_probe(verbose: bool = False) -> str:
    """libusp_probe.so: the plain streaming read the benchmark reports as a reference."""
    tmp = PROBE_LIB + ".tmp"
    cmd = [HIPCC, *DEVICE_FLAGS, "-O3", "-std=c++17", "-fPIC", "-shared", "-Wall",
           os.path.join(CSRC, "usp_probe.hip"), "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed building libusp_probe.so")
    os.replace(tmp, PROBE_LIB)
    return PROBE_LIB


DENSE_LIB = os.path.join(HERE, "libusp_denseref.so")


def build_dense_ref(verbose: bool = False) -> str:
    """libusp_denseref.so: the hipBLASLt dense GEMM the benchmark compares against."""
    tmp = DENSE_LIB + ".tmp"
    cmd = [HIPCC, *DEVICE_FLAGS, "-O2", "-std=c++17", "-fPIC", "-shared", "-Wall",
           os.path.join(CSRC, "usp_dense_ref.cpp"), "-o", tmp, "-lhipblaslt"]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed building libusp_denseref.so")
    os.replace(tmp, DENSE_LIB)
    return DENSE_LIB


if __name__ == "__main__":
    print(build(verbose=True))
