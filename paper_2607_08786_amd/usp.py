"""Python binding of libusp.so: argument marshalling only.

Every function here forwards to the C entry point of the same name declared in
``include/usp.h``; all computation happens in the library's host encoder and
gfx950 kernels. PyTorch supplies device buffers and the current HIP stream.
There is no fallback: if the library is not built, loading it raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch  # imported first so libusp.so binds to the HIP runtime torch already loaded

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libusp.so")

USP_OK = 0
_STATUS = {0: "USP_OK", 1: "USP_ERR_INVALID_ARG", 2: "USP_ERR_UNSUPPORTED", 3: "USP_ERR_OOM",
           4: "USP_ERR_HIP", 5: "USP_ERR_INTERNAL"}

EXPORTED = ("usp_encode", "usp_workspace_size", "usp_spmm", "usp_spmm_ex", "usp_spmm_noalloc", "usp_plan",
            "usp_densify", "usp_decode", "usp_info", "usp_free", "usp_last_error")

# Bytes of the per-GPU device scratch usp_spmm_noalloc uses (USP_NOALLOC_SCRATCH_BYTES).
NOALLOC_SCRATCH_BYTES = 32 << 20

# usp_activation
ACTIVATIONS = {"none": 0, "relu": 1, "gelu_tanh": 2, "silu": 3}


class UspError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{_STATUS.get(status, status)}: {msg}")
        self.status = status


class usp_info_t(ctypes.Structure):
    _fields_ = [("M", ctypes.c_int64), ("K", ctypes.c_int64), ("nnz", ctypes.c_int64),
                ("device_bytes", ctypes.c_size_t), ("table_bytes", ctypes.c_size_t),
                ("format_version", ctypes.c_int32), ("tile_rows", ctypes.c_int32),
                ("tile_k", ctypes.c_int32), ("device", ctypes.c_int32)]


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Loads libusp.so (raises when it has not been built)."""
    global _lib
    if _lib is not None and path == LIB_PATH:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built: run paper_2607_08786_amd/build.py "
                          "(or __graft_entry__.build()) first")
    lib = ctypes.CDLL(path)
    p, i64, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_size_t
    st = ctypes.c_int
    lib.usp_encode.argtypes = [p, i64, p, i64, i64, i64, ctypes.c_int, ctypes.POINTER(p)]
    lib.usp_encode.restype = st
    lib.usp_workspace_size.argtypes = [p, i64]
    lib.usp_workspace_size.restype = sz
    lib.usp_spmm.argtypes = [p, p, i64, p, i64, i64, p, sz, p]
    lib.usp_spmm.restype = st
    lib.usp_spmm_ex.argtypes = [p, p, i64, p, i64, i64, p, p, i64, ctypes.c_int, p, sz, p]
    lib.usp_spmm_ex.restype = st
    lib.usp_spmm_noalloc.argtypes = [p, p, i64, p, i64, i64, p]
    lib.usp_spmm_noalloc.restype = st
    lib.usp_plan.argtypes = [p, i64, ctypes.c_char_p, sz]
    lib.usp_plan.restype = st
    lib.usp_densify.argtypes = [p, p, i64, p]
    lib.usp_densify.restype = st
    lib.usp_decode.argtypes = [p, p, p]
    lib.usp_decode.restype = st
    lib.usp_info.argtypes = [p, ctypes.POINTER(usp_info_t)]
    lib.usp_info.restype = st
    lib.usp_free.argtypes = [p]
    lib.usp_free.restype = st
    lib.usp_last_error.argtypes = []
    lib.usp_last_error.restype = ctypes.c_char_p
    if path == LIB_PATH:
        _lib = lib
    return lib


def usp_last_error() -> str:
    return load_library().usp_last_error().decode()


def _check(status: int):
    if status != USP_OK:
        raise UspError(status, usp_last_error())


def _torch_stream(stream):
    """The torch stream a call is enqueued on: the current one, a torch.cuda.Stream, or a raw
    hipStream_t handle wrapped as an external stream."""
    if stream is None:
        return torch.cuda.current_stream()
    if isinstance(stream, torch.cuda.Stream):
        return stream
    return torch.cuda.ExternalStream(int(stream))


def _stream_handle(stream) -> int | None:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def usp_encode(W: np.ndarray, mask: np.ndarray, device: int = 0) -> int:
    """W: (M, K) fp16 bit patterns (uint16 or float16); mask: (M, K), nonzero = kept."""
    W = np.ascontiguousarray(W)
    if W.dtype == np.float16:
        W = W.view(np.uint16)
    if W.dtype != np.uint16 or W.ndim != 2:
        raise TypeError("W must be a 2-D uint16 (fp16 bits) or float16 array")
    mask = np.ascontiguousarray(mask)
    if mask.dtype == np.bool_:
        mask = mask.view(np.uint8)
    if mask.dtype != np.uint8 or mask.shape != W.shape:
        raise TypeError("mask must be a uint8/bool array of W's shape")
    M, K = W.shape
    h = ctypes.c_void_p()
    _check(load_library().usp_encode(W.ctypes.data, K, mask.ctypes.data, K, M, K, device, ctypes.byref(h)))
    return h.value


def usp_workspace_size(handle: int, N: int) -> int:
    return int(load_library().usp_workspace_size(handle, N))


def usp_plan(handle: int, N: int) -> str:
    """The kernel usp_spmm runs for this handle and N (X aligned, ldx = K), as text."""
    buf = ctypes.create_string_buffer(128)
    _check(load_library().usp_plan(handle, N, buf, len(buf)))
    return buf.value.decode()


def usp_spmm(handle: int, X: torch.Tensor, Y: torch.Tensor, workspace: torch.Tensor | None = None,
             stream=None) -> None:
    """Y[N, M] = X[N, K] @ W^T, i.e. Y = W X with token-major X and Y (fp16 device tensors)."""
    if X.dtype != torch.float16 or Y.dtype != torch.float16:
        raise TypeError("X and Y must be float16")
    if X.dim() != 2 or Y.dim() != 2 or X.stride(1) != 1 or Y.stride(1) != 1:
        raise TypeError("X and Y must be 2-D with unit inner stride")
    N = X.shape[0]
    if Y.shape[0] != N:
        raise ValueError("X and Y must have the same number of tokens")
    ws_ptr, ws_bytes = None, 0
    if workspace is not None:
        ws_ptr, ws_bytes = workspace.data_ptr(), workspace.numel() * workspace.element_size()
    _check(load_library().usp_spmm(handle, X.data_ptr(), X.stride(0), Y.data_ptr(), Y.stride(0), N,
                                   ws_ptr, ws_bytes, _stream_handle(stream)))


def usp_spmm_ex(handle: int, X: torch.Tensor, Y: torch.Tensor, workspace: torch.Tensor | None = None,
                bias: torch.Tensor | None = None, residual: torch.Tensor | None = None,
                activation: str | int = "none", stream=None) -> None:
    """Y = act(X @ W^T + bias) + residual (token-major fp16 device tensors; bias [M],
    residual [N, M] with unit inner stride, or None; residual may be Y itself)."""
    if X.dtype != torch.float16 or Y.dtype != torch.float16:
        raise TypeError("X and Y must be float16")
    if X.dim() != 2 or Y.dim() != 2 or X.stride(1) != 1 or Y.stride(1) != 1:
        raise TypeError("X and Y must be 2-D with unit inner stride")
    N = X.shape[0]
    if Y.shape[0] != N:
        raise ValueError("X and Y must have the same number of tokens")
    act = ACTIVATIONS[activation] if isinstance(activation, str) else int(activation)
    b_ptr = r_ptr = None
    ldr = 0
    if bias is not None:
        if bias.dtype != torch.float16 or bias.dim() != 1 or bias.stride(0) != 1 or bias.shape[0] != Y.shape[1]:
            raise TypeError("bias must be a contiguous float16 vector of M entries")
        b_ptr = bias.data_ptr()
    if residual is not None:
        if residual.dtype != torch.float16 or residual.dim() != 2 or residual.stride(1) != 1 \
                or tuple(residual.shape) != tuple(Y.shape):
            raise TypeError("residual must be a float16 [N, M] tensor with unit inner stride")
        r_ptr, ldr = residual.data_ptr(), residual.stride(0)
    ws_ptr, ws_bytes = None, 0
    if workspace is not None:
        ws_ptr, ws_bytes = workspace.data_ptr(), workspace.numel() * workspace.element_size()
    _check(load_library().usp_spmm_ex(handle, X.data_ptr(), X.stride(0), Y.data_ptr(), Y.stride(0), N,
                                      b_ptr, r_ptr, ldr, act, ws_ptr, ws_bytes, _stream_handle(stream)))


def usp_spmm_noalloc(handle: int, X: torch.Tensor, Y: torch.Tensor, stream=None) -> None:
    """usp_spmm with the library's per-GPU device scratch as its workspace (no allocation;
    calls overlapping on one GPU must be serialized by the caller)."""
    if X.dtype != torch.float16 or Y.dtype != torch.float16:
        raise TypeError("X and Y must be float16")
    if X.dim() != 2 or Y.dim() != 2 or X.stride(1) != 1 or Y.stride(1) != 1:
        raise TypeError("X and Y must be 2-D with unit inner stride")
    N = X.shape[0]
    if Y.shape[0] != N:
        raise ValueError("X and Y must have the same number of tokens")
    _check(load_library().usp_spmm_noalloc(handle, X.data_ptr(), X.stride(0), Y.data_ptr(), Y.stride(0), N,
                                           _stream_handle(stream)))


def usp_densify(handle: int, Wd: torch.Tensor, stream=None) -> None:
    if Wd.dtype != torch.float16 or Wd.dim() != 2 or Wd.stride(1) != 1:
        raise TypeError("Wd must be a 2-D float16 tensor with unit inner stride")
    _check(load_library().usp_densify(handle, Wd.data_ptr(), Wd.stride(0), _stream_handle(stream)))


def usp_info(handle: int) -> dict:
    info = usp_info_t()
    _check(load_library().usp_info(handle, ctypes.byref(info)))
    return {f: getattr(info, f) for f, _ in usp_info_t._fields_}


def usp_decode(handle: int):
    info = usp_info(handle)
    M, K = info["M"], info["K"]
    W = np.empty((M, K), dtype=np.uint16)
    mask = np.empty((M, K), dtype=np.uint8)
    _check(load_library().usp_decode(handle, W.ctypes.data, mask.ctypes.data))
    return W, mask


def usp_free(handle: int) -> None:
    _check(load_library().usp_free(handle))


class SparseMatrix:
    """Owns one encoded weight matrix (a usp_matrix handle)."""

    def __init__(self, W: np.ndarray, mask: np.ndarray, device: int = 0):
        self.handle = usp_encode(W, mask, device)
        info = usp_info(self.handle)
        self.M, self.K, self.nnz = info["M"], info["K"], info["nnz"]
        self.device = device
        self.device_bytes = info["device_bytes"] + info["table_bytes"]

    def workspace_size(self, N: int) -> int:
        return usp_workspace_size(self.handle, N)

    def plan(self, N: int) -> str:
        return usp_plan(self.handle, N)

    def make_workspace(self, N: int, stream=None) -> torch.Tensor | None:
        """A zero-filled workspace for N tokens, allocated and cleared on `stream` (default: the
        current stream), so calls enqueued on that stream are ordered after the clear."""
        n = self.workspace_size(N)
        if n == 0:
            return None
        with torch.cuda.stream(_torch_stream(stream)):
            return torch.zeros(n, dtype=torch.uint8, device=f"cuda:{self.device}")  # zeroed once

    def spmm(self, X: torch.Tensor, Y: torch.Tensor | None = None, workspace=None, stream=None,
             bias: torch.Tensor | None = None, residual: torch.Tensor | None = None,
             activation: str | int = "none") -> torch.Tensor:
        """Y = W X (token-major), or act(W X + bias) + residual when any of those is given.

        A Y or workspace this call creates is allocated on `stream`, the stream the product is
        enqueued on, so the caching allocator only reuses that memory in that stream's order."""
        N = X.shape[0]
        if Y is None or workspace is None:
            with torch.cuda.stream(_torch_stream(stream)):
                if Y is None:
                    Y = torch.empty((N, self.M), dtype=torch.float16, device=X.device)
                if workspace is None:
                    workspace = self.make_workspace(N)
        if bias is None and residual is None and activation in ("none", 0):
            usp_spmm(self.handle, X, Y, workspace, stream)
        else:
            usp_spmm_ex(self.handle, X, Y, workspace, bias, residual, activation, stream)
        return Y

    def densify(self, stream=None) -> torch.Tensor:
        Wd = torch.empty((self.M, self.K), dtype=torch.float16, device=f"cuda:{self.device}")
        usp_densify(self.handle, Wd, stream)
        return Wd

    def decode(self):
        return usp_decode(self.handle)

    def info(self) -> dict:
        return usp_info(self.handle)

    def free(self) -> None:
        if self.handle:
            usp_free(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass
