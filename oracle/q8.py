"""fp64 CPU oracle for the Q8_0 matrix-vector product (decode linear layers).

TEST INFRASTRUCTURE ONLY: the test suite, the package smoke check and the
benchmark's CPU-baseline leg may import this module; the product library and
its Python binding never do.  It shares no code with the GPU path.

The arithmetic lives in ``q8_oracle.c`` (plain C, double precision, one
thread, no fast-math, no contraction); this module builds it with gcc, loads
it with ctypes and converts inputs exactly to float64.

Definition followed (Sec. 4.3, linear layers as GEMV in decode; Q8_0 blocks
of one binary16 scale and 32 int8 values, the scale first as in Sec. 7):
y[m] = sum_b sum_j d[m, b] * q[m, b, j] * x[32 b + j].
Layout: w is uint8 [M, K / 32, 34] (bytes 0-1 the little-endian scale, bytes
2-33 the int8 values), x [K], y [M].
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "q8_oracle.c")
_LIB = os.path.join(_HERE, "libq8oracle.so")
_lib = None

_DP = ctypes.POINTER(ctypes.c_double)
_BP = ctypes.POINTER(ctypes.c_uint8)


def build(force: bool = False) -> str:
    """Compile q8_oracle.c into libq8oracle.so with gcc (strict IEEE double)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-fPIC", "-shared", "-std=c11", "-ffp-contract=off",
               "-fno-fast-math", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB)
        lib.q8_half_to_f64.argtypes = [ctypes.c_uint]
        lib.q8_half_to_f64.restype = ctypes.c_double
        lib.q8_0_gemv_f64.argtypes = [_BP, _DP, _DP, ctypes.c_int, ctypes.c_int]
        lib.q8_0_gemv_f64.restype = ctypes.c_int
        _lib = lib
    return _lib


def half_to_f64(bits: int) -> float:
    """The oracle's binary16 decoding of one 16-bit pattern."""
    return float(_load().q8_half_to_f64(int(bits) & 0xFFFF))


def gemv(w, x) -> np.ndarray:
    """y = W x in float64 for Q8_0 weights ``w`` (uint8 [M, K/32, 34], or
    [M, K/32 * 34]) and activations ``x`` (any real dtype, length K)."""
    w = np.ascontiguousarray(np.asarray(w, dtype=np.uint8))
    M = w.shape[0]
    xb = np.ascontiguousarray(np.asarray(x, dtype=np.float64).reshape(-1))
    K = xb.shape[0]
    if w.size != M * (K // 32) * 34:
        raise ValueError("w must hold M rows of K/32 blocks of 34 bytes")
    y = np.empty(M, dtype=np.float64)
    st = _load().q8_0_gemv_f64(w.ctypes.data_as(_BP), xb.ctypes.data_as(_DP),
                               y.ctypes.data_as(_DP), M, K)
    if st != 0:
        raise ValueError("oracle rejected the arguments")
    return y
