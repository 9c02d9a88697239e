"""Builds and loads the host-only encoder harness (tests/native) with g++."""
import ctypes
import os
import subprocess

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = [os.path.join(ROOT, "tests", "native", "encode_host_test.cpp"),
       os.path.join(ROOT, "paper_2607_08786_amd", "csrc", "usp_encode.cpp")]


def build(out_dir: str, sanitize: bool = False) -> ctypes.CDLL:
    out = os.path.join(out_dir, "libusp_host_test%s.so" % ("_asan" if sanitize else ""))
    cmd = ["g++", "-O1" if sanitize else "-O2", "-g", "-std=c++17", "-fPIC", "-shared",
           "-I", os.path.join(ROOT, "include"), *SRC, "-o", out, "-lpthread"]
    if sanitize:
        cmd[1:1] = ["-fsanitize=address,undefined", "-fno-omit-frame-pointer"]
    subprocess.run(cmd, check=True)
    lib = ctypes.CDLL(out)
    p, i64 = ctypes.c_void_p, ctypes.c_int64
    lib.usp_test_roundtrip.argtypes = [p, i64, p, i64, i64, i64, p, p, p, p, p]
    lib.usp_test_roundtrip.restype = ctypes.c_int
    lib.usp_test_records.argtypes = [p, p, i64, i64, p, p]
    lib.usp_test_records.restype = ctypes.c_int
    return lib


def roundtrip(lib, W: np.ndarray, mask: np.ndarray):
    W = np.ascontiguousarray(W, dtype=np.uint16)
    mask = np.ascontiguousarray(mask, dtype=np.uint8)
    M, K = W.shape
    Wo = np.empty_like(W)
    mo = np.empty_like(mask)
    nnz, sb, tiles = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    rc = lib.usp_test_roundtrip(W.ctypes.data, K, mask.ctypes.data, K, M, K, Wo.ctypes.data, mo.ctypes.data,
                                ctypes.byref(nnz), ctypes.byref(sb), ctypes.byref(tiles))
    assert rc == 0, rc
    return Wo, mo, nnz.value, sb.value, tiles.value
