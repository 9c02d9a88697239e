"""C ABI checks that need no GPU: the library loads, exports every entry point
include/usp.h declares, and rejects bad arguments before touching a device."""
import ctypes
import os
import re
import threading

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "usp.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(usp_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def usp():
    from paper_2607_08786_amd import usp as mod
    return mod


def test_header_declares_the_binding_surface(usp):
    assert declared_functions() == sorted(usp.EXPORTED)


def test_library_exports_every_declared_symbol(usp):
    lib = usp.load_library()
    for name in declared_functions():
        assert hasattr(lib, name), name
    out = os.popen(f"nm -D --defined-only {usp.LIB_PATH}").read()
    for name in declared_functions():
        assert re.search(rf"\bT {name}\b", out), name


def test_argument_errors_without_device(usp):
    lib = usp.load_library()
    p = ctypes.c_void_p
    assert lib.usp_free(None) == 0
    assert lib.usp_workspace_size(None, 16) == 0
    buf = ctypes.create_string_buffer(64)
    assert lib.usp_plan(None, 16, buf, 64) == 1
    info = usp.usp_info_t()
    assert lib.usp_info(None, ctypes.byref(info)) == 1
    assert "invalid" in usp.usp_last_error()
    assert lib.usp_spmm(None, None, 0, None, 0, 16, None, 0, None) == 1
    h = p()
    assert lib.usp_encode(None, 4, None, 4, 4, 4, 0, ctypes.byref(h)) == 1 and h.value is None
    buf = (ctypes.c_uint16 * 16)()
    mb = (ctypes.c_uint8 * 16)()
    assert lib.usp_encode(buf, 4, mb, 4, 0, 4, 0, ctypes.byref(h)) == 1  # M < 1
    assert lib.usp_encode(buf, 3, mb, 4, 4, 4, 0, ctypes.byref(h)) == 1  # ldw < K
    assert "ldw" in usp.usp_last_error()
    assert lib.usp_densify(None, None, 0, None) == 1
    assert lib.usp_decode(None, None, None) == 1
    # More than 2^20 rows: refused before W or the mask is read.
    assert lib.usp_encode(buf, 4, mb, 4, (1 << 20) + 1, 4, 0, ctypes.byref(h)) == 2
    assert "2^20" in usp.usp_last_error() and h.value is None


def test_unknown_handles_are_rejected_without_being_read(usp):
    """A pointer usp_encode never returned (here: ordinary host memory holding
    garbage) is looked up, not dereferenced: every entry point says invalid."""
    lib = usp.load_library()
    junk = ctypes.create_string_buffer(b"\xff" * 512)
    fake = ctypes.cast(junk, ctypes.c_void_p)
    info = usp.usp_info_t()
    assert lib.usp_info(fake, ctypes.byref(info)) == 1
    assert lib.usp_workspace_size(fake, 16) == 0
    assert lib.usp_spmm(fake, fake, 8, fake, 8, 16, None, 0, None) == 1
    assert lib.usp_free(fake) == 1 and "freed" in usp.usp_last_error()


def test_last_error_is_thread_local(usp):
    lib = usp.load_library()
    lib.usp_spmm(None, None, 0, None, 0, 16, None, 0, None)
    assert usp.usp_last_error() != ""
    seen = []
    t = threading.Thread(target=lambda: seen.append(usp.usp_last_error()))
    t.start()
    t.join()
    assert seen == [""]


def test_sparse_linear_op_is_registered():
    # The custom operator exists and its fake (meta) implementation gives the
    # output shape without a device.
    import torch
    from torch._subclasses.fake_tensor import FakeTensorMode
    import paper_2607_08786_amd.linear  # noqa: F401
    with FakeTensorMode():
        x = torch.empty(7, 64, dtype=torch.float16)
        y = torch.ops.usp.sparse_linear(x, 0, 33, None, None, 1, None)
    assert tuple(y.shape) == (7, 33) and y.dtype == torch.float16


# The benchmark's streaming-read reference library builds and exports its entry
# point (no GPU call here).
def test_probe_library_exports_read():
    import ctypes
    import os
    path = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2607_08786_amd",
                        "libusp_probe.so")
    lib = ctypes.CDLL(path)
    assert hasattr(lib, "usp_probe_read")
