"""CPU oracle -- TEST INFRASTRUCTURE ONLY.

Python access to ``oracle.c`` (plain C, float64): the masked dense product that
the sparse kernel must reproduce, and the masked fp16 bit patterns that an
encode/decode round trip must reproduce. Only ``tests/``, the smoke check in
``__graft_entry__`` and the CPU-baseline leg of ``bench.py`` use this module.
It shares no code with the GPU path.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIBS: dict = {}


def lib_path(mutant: int = 0, out_dir: str | None = None) -> str:
    name = "liboracle.so" if mutant == 0 else f"liboracle_mutant{mutant}.so"
    return os.path.join(out_dir or _HERE, name)


def build(mutant: int = 0, out_dir: str | None = None) -> str:
    """Compile oracle.c with gcc (OpenMP over output rows). Returns the .so path."""
    out = lib_path(mutant, out_dir)
    tmp = out + ".tmp"
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99", "-Wall",
           f"-DORACLE_MUTANT={mutant}", _SRC, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def load(mutant: int = 0, out_dir: str | None = None) -> ctypes.CDLL:
    key = (mutant, out_dir)
    if key in _LIBS:
        return _LIBS[key]
    path = lib_path(mutant, out_dir)
    if not os.path.exists(path) or (mutant == 0 and os.path.getmtime(path) < os.path.getmtime(_SRC)):
        build(mutant, out_dir)
    lib = ctypes.CDLL(path)
    p = ctypes.c_void_p
    i64 = ctypes.c_int64
    lib.oracle_f16_to_f64.restype = ctypes.c_double
    lib.oracle_f16_to_f64.argtypes = [ctypes.c_uint16]
    lib.oracle_f16_to_f64_array.restype = None
    lib.oracle_f16_to_f64_array.argtypes = [p, i64, p]
    lib.oracle_num_threads.restype = ctypes.c_int
    lib.oracle_num_threads.argtypes = []
    lib.oracle_masked_gemm_rows.restype = ctypes.c_int
    lib.oracle_masked_gemm_rows.argtypes = [p, i64, p, i64, p, i64, i64, i64, i64, p, i64, p, p]
    lib.oracle_masked_bits.restype = None
    lib.oracle_masked_bits.argtypes = [p, i64, p, i64, i64, i64, p]
    _LIBS[key] = lib
    return lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def f16_to_f64(bits: np.ndarray, lib=None) -> np.ndarray:
    lib = lib or load()
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    out = np.empty(b.shape, dtype=np.float64)
    lib.oracle_f16_to_f64_array(_ptr(b), b.size, _ptr(out))
    return out


def masked_gemm(W: np.ndarray, mask: np.ndarray, X: np.ndarray, rows=None, lib=None):
    """Y, A as float64 arrays of shape (N, R): Y[n, i] = sum_k kept W[rows[i], k] * X[n, k].

    W: (M, K) uint16 fp16 bits; mask: (M, K) uint8; X: (N, K) uint16 fp16 bits
    (token-major). ``rows`` selects output rows (default: all, in order).
    """
    lib = lib or load()
    W = np.ascontiguousarray(W, dtype=np.uint16)
    mask = np.ascontiguousarray(mask, dtype=np.uint8)
    X = np.ascontiguousarray(X, dtype=np.uint16)
    M, K = W.shape
    N = X.shape[0]
    assert mask.shape == (M, K) and X.shape == (N, K)
    if rows is None:
        R = M
        rows_p = None
    else:
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        R = rows.size
        rows_p = _ptr(rows)
    Y = np.empty((N, R), dtype=np.float64)
    A = np.empty((N, R), dtype=np.float64)
    rc = lib.oracle_masked_gemm_rows(_ptr(W), K, _ptr(mask), K, _ptr(X), K, M, K, N,
                                     rows_p, R, _ptr(Y), _ptr(A))
    if rc != 0:
        raise ValueError("oracle_masked_gemm_rows rejected its arguments")
    return Y, A


def masked_bits(W: np.ndarray, mask: np.ndarray, lib=None) -> np.ndarray:
    lib = lib or load()
    W = np.ascontiguousarray(W, dtype=np.uint16)
    mask = np.ascontiguousarray(mask, dtype=np.uint8)
    M, K = W.shape
    out = np.empty((M, K), dtype=np.uint16)
    lib.oracle_masked_bits(_ptr(W), K, _ptr(mask), K, M, K, _ptr(out))
    return out


# Fused linear-layer epilogue: Y = act(W X + bias) + residual (float64).
ACTIVATIONS = {"none": 0, "relu": 1, "gelu_tanh": 2, "silu": 3}
# Largest slope of each activation (a bound used to carry the product's error
# through it): 1 for the identity and ReLU; the tanh form of GELU peaks at
# ~1.129 and SiLU at ~1.100.
ACT_SLOPE_BOUND = 1.13


def activation(v: np.ndarray, act: int) -> np.ndarray:
    """ReLU: max(v, 0). GELU, tanh form: v/2 * (1 + tanh(sqrt(2/pi) (v + 0.044715 v^3))).
    SiLU: v / (1 + exp(-v))."""
    v = np.asarray(v, dtype=np.float64)
    if act == 0:
        return v
    if act == 1:
        return np.maximum(v, 0.0)
    if act == 2:
        return 0.5 * v * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (v + 0.044715 * v ** 3)))
    if act == 3:
        with np.errstate(over="ignore"):
            return v / (1.0 + np.exp(-v))
    raise ValueError(f"unknown activation {act}")


def linear_epilogue(Yref: np.ndarray, A: np.ndarray, act: int, bias=None, residual=None):
    """The product's reference (Yref, A of shape (N, R)) through the epilogue:
    Y = act(Yref + bias) + residual, and the scale its error is bounded by,
    A' = L (A + |bias|) + |residual| (L = 1 without an activation's slope).
    bias: float64 [R] or None; residual: float64 (N, R) or None."""
    z = Yref + (0.0 if bias is None else bias[None, :])
    y = activation(z, act)
    scale = A + (0.0 if bias is None else np.abs(bias)[None, :])
    if act in (2, 3):
        scale = ACT_SLOPE_BOUND * scale
    if residual is not None:
        y = y + residual
        scale = scale + np.abs(residual)
    return y, scale


def num_threads(lib=None) -> int:
    return int((lib or load()).oracle_num_threads())


def check_tolerance(Y: np.ndarray, Yref: np.ndarray, A: np.ndarray,
                    rel: float = 1e-2, abs_: float = 1e-3, frob: float = 1e-3) -> dict:
    """Acceptance test of a computed Y (float64 view of the fp16 output) against the oracle.

    Elementwise |Y - Yref| <= rel * A + abs_, and relative Frobenius error <= frob
    (when Yref is identically zero, Y must be identically zero).
    """
    Y = np.asarray(Y, dtype=np.float64)
    err = np.abs(Y - Yref)
    bound = rel * A + abs_
    ok_elem = bool(np.all(err <= bound))
    nref = float(np.linalg.norm(Yref))
    if nref == 0.0:
        frob_err = float(np.linalg.norm(Y))
        ok_frob = frob_err == 0.0
    else:
        frob_err = float(np.linalg.norm(Y - Yref) / nref)
        ok_frob = frob_err <= frob
    worst = float(np.max(err / bound)) if err.size else 0.0
    return dict(ok=ok_elem and ok_frob, ok_elem=ok_elem, ok_frob=ok_frob,
                frob_err=frob_err, worst_ratio=worst)
