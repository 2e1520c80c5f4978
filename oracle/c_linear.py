"""ctypes binding of the plain-C fp64 linear oracle (oracle/c/q4_linear.c).

TEST INFRASTRUCTURE ONLY: used by the test suite and by the benchmark's
CPU-baseline leg; it shares no code with the HIP library.  build() compiles
the C source with gcc into oracle/c/liboracle_q4.so.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c")
SRC = os.path.join(_HERE, "q4_linear.c")
LIB = os.path.join(_HERE, "liboracle_q4.so")
_lib = None


def build() -> str:
    tmp = LIB + f".tmp{os.getpid()}"
    subprocess.run(["gcc", "-O2", "-std=c99", "-Wall", "-shared", "-fPIC", "-pthread", "-o", tmp, SRC, "-lm"],
                   check=True, capture_output=True, text=True)
    os.replace(tmp, LIB)
    return LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build()
        l = ctypes.CDLL(LIB)
        l.q4_linear_f64.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                    ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int]
        l.q4_linear_f64.restype = ctypes.c_int
        _lib = l
    return _lib


def linear(x, codes, scales, threads: int = 1) -> np.ndarray:
    """y[M][N] in fp64 from fp16 (or any float) x[M][K], codes uint8[N][K/2], fp16 scales[N][K/32]."""
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    sbits = np.ascontiguousarray(np.asarray(scales, dtype=np.float16)).view(np.uint16)
    xd = np.ascontiguousarray(np.asarray(x, dtype=np.float64).reshape(-1, 2 * codes.shape[1]))
    N, K, M = codes.shape[0], 2 * codes.shape[1], xd.shape[0]
    y = np.empty((M, N), dtype=np.float64)
    rc = _load().q4_linear_f64(codes.ctypes.data, sbits.ctypes.data, N, K, xd.ctypes.data, M, y.ctypes.data,
                               int(threads))
    if rc != 0:
        raise ValueError("q4_linear_f64 rejected its arguments")
    return y
