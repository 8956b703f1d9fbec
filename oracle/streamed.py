"""Float32 oracle over bf16 weights kept as bit patterns (test infrastructure
only, like the rest of ``oracle/``).

The 32B-shaped decoder has 33e9 weight parameters: 133 GB in float32, more
than the host that writes the full-depth references holds.  This model runs
the same decoder forward (``oracle.model.forward``, §3.1 Verify with the
unchanged target) with every linear layer computed from the bf16 bit patterns
directly: ``oracle_gemv_bf16`` in ``gemv_bf16.c`` widens each weight exactly
and multiplies in float32, for inputs of up to ``gemv_rows`` rows; larger
inputs (a prefill) widen the whole matrix to float32 and use numpy's product.
Either way y = h W^T with every weight taken exactly and float32 arithmetic,
so results agree with ``OracleModel(dtype=float32)`` up to float32 summation
order (pinned in tests/test_oracle_streamed.py).
"""

import ctypes
import os
import subprocess

import numpy as np

from .model import OracleModel, bf16_bits_to_float

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "gemv_bf16.c")
LIB = os.path.join(HERE, "liboracle_gemv.so")

_lib = None


def build_gemv() -> str:
    """Compile gemv_bf16.c (plain C, OpenMP) next to this file."""
    tmp = LIB + ".tmp"
    subprocess.run(["gcc", "-O3", "-march=native", "-fopenmp", "-fPIC", "-shared", SRC, "-o", tmp],
                   check=True)
    os.replace(tmp, LIB)
    return LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build_gemv()
        lib = ctypes.CDLL(LIB)
        lib.oracle_gemv_bf16.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
                                         ctypes.c_int64, ctypes.c_void_p]
        lib.oracle_gemv_bf16.restype = None
        _lib = lib
    return _lib


def gemv_bf16(h: np.ndarray, w_bits: np.ndarray) -> np.ndarray:
    """h [M, K] float32 times the transpose of the bf16 matrix w_bits [N, K]."""
    h = np.ascontiguousarray(h, dtype=np.float32)
    w = np.ascontiguousarray(w_bits, dtype=np.uint16)
    M, K = h.shape
    N, K2 = w.shape
    assert K == K2, (h.shape, w.shape)
    y = np.empty((M, N), dtype=np.float32)
    _load().oracle_gemv_bf16(h.ctypes.data, M, w.ctypes.data, N, K, y.ctypes.data)
    return y


class StreamedOracleModel(OracleModel):
    """float32 oracle whose weight mapping may fetch each tensor on demand
    (from memory, a file or its seed); nothing converted is kept."""

    def __init__(self, cfg, weights, gemv_rows: int = 256):
        super().__init__(cfg, weights, dtype=np.float32, cache=False)
        self.gemv_rows = gemv_rows

    def linear(self, h, name):
        w = self.weights[name]
        h = np.asarray(h, dtype=np.float32)
        if h.shape[0] <= self.gemv_rows:
            return gemv_bf16(h, w)
        return h @ bf16_bits_to_float(w, np.float32).T
