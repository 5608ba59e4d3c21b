"""Build and binding of the test-side sparse-MFMA consumer
(tests/sparse_mfma_check.hip): a 2:4-sparse bf16 product on gfx950's sparse
matrix core that reads the export's compressed values and metadata as they are
written.  Built by ``__graft_entry__.build()`` next to the library; the GPU test
that uses it fails when it is missing."""
from __future__ import annotations

import ctypes
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "sparse_mfma_check.hip")
LIB_PATH = os.path.join(HERE, "libsparse_mfma_check.so")

_lib = None


def build(verbose: bool = False) -> str:
    from paper_2608_23048_amd.build import HIPCC_FLAGS, hipcc
    tmp = f"{LIB_PATH}.tmp{os.getpid()}"
    cmd = [hipcc(), *HIPCC_FLAGS, SRC, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        L.sparse_check_matmul_2of4.restype = ctypes.c_int
        L.sparse_check_matmul_2of4.argtypes = [ctypes.c_void_p] * 4 + [ctypes.c_int64] * 3 + \
            [ctypes.c_void_p]
        _lib = L
    return _lib


def matmul_2of4(vals, meta, X, rows: int, cols: int):
    """Y [rows, tokens] fp32 = W_sparse X^T from the export's ``vals``
    [rows * cols / 4, 2] bf16 and ``meta`` words; X [tokens, cols] bf16."""
    import torch
    tokens = X.shape[0]
    assert X.dtype == torch.bfloat16 and X.is_contiguous() and X.shape[1] == cols
    assert vals.dtype == torch.bfloat16 and vals.is_contiguous() and vals.numel() == rows * cols // 2
    assert meta.is_contiguous() and meta.numel() * 32 >= rows * cols
    assert meta.element_size() == 4 and vals.device == X.device == meta.device
    Y = torch.empty((rows, tokens), dtype=torch.float32, device=X.device)
    stream = torch.cuda.current_stream(X.device).cuda_stream
    rc = lib().sparse_check_matmul_2of4(vals.data_ptr(), meta.data_ptr(), X.data_ptr(),
                                        Y.data_ptr(), rows, cols, tokens, stream)
    if rc != 0:
        raise RuntimeError(f"sparse_check_matmul_2of4 failed ({rc})")
    return Y
