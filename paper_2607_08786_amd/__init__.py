"""MI355X-native unstructured-sparse fp16 SpMM (decode-phase Y = W X).

The C ABI lives in ``include/usp.h`` and ``libusp.so``; ``usp`` is its Python
binding. Importing this package does not load the library; the first call does,
and raises if it has not been built.
"""
from . import usp  # noqa: F401
from .usp import (  # noqa: F401
    SparseMatrix,
    UspError,
    load_library,
    usp_decode,
    usp_densify,
    usp_encode,
    usp_free,
    usp_info,
    usp_last_error,
    usp_spmm,
    usp_workspace_size,
)
